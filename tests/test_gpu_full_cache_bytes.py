"""Every byte of every full-size low-bit cache against the oracle's packing (GPU).

The default suite compares the GPU-written pages of sampled sequences at full
size (``test_gpu_decode.py``).  This test compares all of them: every token
of every sequence of each full-size configuration and of the 64 x 32768
shape, written by the step the benchmark times (prefill through
``mla_lowbit_quant_append``, the step's tokens appended inside the decode
launch), region by region against the oracle's quantize-and-pack of the same
tokens (Appendix C.4, "Affine group quantization").  The oracle's packing of
the 10.8M tokens takes minutes of host time on one core, so it runs in 16
worker processes (started fresh, no GPU use), each returning a digest per
sequence; about a minute in all.
"""
import hashlib
import multiprocessing as mp
import time

import numpy as np
import pytest

from gpu_support import gpu_pages, oracle_format
from oracle import paged_cache as pc
from paper_2609_36760_amd import synthetic as syn

pytestmark = pytest.mark.gpu

CONFIGS = [
    # (workload, layer)
    ("tiny_b1_h16_256", 0),
    ("dsv3_b32_h128_4k_c4r4", 0),
    ("int2_b64_h128_32k_c2r4", 0),
    ("splitkv_b8_h128_128k_c4r4", 0),
    ("ragged_b96_h128_sq2_mixed", 0),
    ("ragged_b96_h128_sq2_mixed", 1),
    ("c4r4_b64_h128_32k", 0),
]


def _digest(blocks):
    h = hashlib.sha256()
    for blk in blocks:
        h.update(np.ascontiguousarray(blk).tobytes())
    return h.hexdigest()


def oracle_digest(job):
    """Worker: the oracle's packing of sequence b (its L tokens), hashed."""
    name, layer, b, L, c_bits, r_bits, meta = job
    c, k = syn.sequence_tokens(syn.WORKLOADS[name], layer, b, L)
    return b, _digest(pc.encode_tokens(pc.CacheFormat(c_bits=c_bits, r_bits=r_bits, meta=meta), c, k))


@pytest.mark.parametrize("config", CONFIGS, ids=[f"{n}-L{l}" for n, l in CONFIGS])
def test_full_cache_bytes(config):
    import torch

    from paper_2609_36760_amd.runner import DecodeRun
    name, layer = config
    t0 = time.perf_counter()
    run = DecodeRun(syn.WORKLOADS[name], layer=layer)
    run.fused_step()
    torch.cuda.synchronize()
    fmt = oracle_format(run)
    lens = [int(x) for x in run.lens]
    jobs = [(name, layer, b, L, run.c_bits, run.r_bits, run.meta) for b, L in enumerate(lens)]
    with mp.get_context("spawn").Pool(16) as pool:
        want = dict(pool.map(oracle_digest, jobs, chunksize=1))
    bad = []
    for b, L in enumerate(lens):
        if _digest(pc.page_blocks(fmt, gpu_pages(run, b), L)) != want[b]:
            bad.append(b)
    tokens = sum(lens)
    print(f"{name} layer {layer}: {len(lens)} sequences, {tokens} tokens, "
          f"{tokens * sum(fmt.region_sizes())} cache bytes compared, {len(bad)} sequences differ, "
          f"{time.perf_counter() - t0:.1f} s", flush=True)
    assert not bad, f"{name} layer {layer}: sequences whose bytes differ from the oracle's packing: {bad[:10]}"
