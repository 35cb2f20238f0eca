"""CPU oracle for low-bit MLA decode -- TEST INFRASTRUCTURE ONLY.

This package is the plain, slow, obviously-correct definition of what the
GPU path computes.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it.  The product library
(``paper_2609_36760_amd``) never imports, links or executes anything here,
and nothing here imports the product library: the two share no code.

Modules
-------
``quantizer``   affine asymmetric per-token group quantizer, integer packing,
                dequantization (Appendix C.4, "Affine group quantization").
                fp32 arithmetic in the paper's order, round-half-to-even.
``paged_cache`` the byte layout of one packed cache page and the slot-mapped
                insertion of tokens (Appendix C.5, "Cache update and tile
                reuse", "Storage layout"); also reads a page back.
``attention``   absorbed dual-path MLA attention in fp64 (Sec. 2.1,
                eq. mla_compact), chunk partials and their global-normalisation
                merge (Appendix C.5, "Global attention normalization").
``reference_mla`` the materialised, non-absorbed MLA head computation and the
                positional-QK output bound (Sec. 2.1; Sec. 3.2,
                Proposition 2, proved in Appendix C.3), used only to pin
                ``attention``.
``storage``     per-layer persistent storage accounting
                (Appendix C.5, eq. physical_cache_storage).

Every function is pinned by ``tests/test_oracle_*.py`` against values the
paper fixes, closed forms, invariants or brute force on tiny inputs.
"""
