"""Which work item writes a new token inside a protected decode launch (host
logic of the in-launch writer; no GPU).

Under BF16 protection (Appendix C.5, "BF16 protection and cache lifecycle")
a sequence's keys form a list of 32-token tiles: the packed tiles from the
tile holding token `sink` up to position L - recent, then the protected rows
in position order (the sink rows, then the recent window).  A key split
takes a contiguous range of that list.  The decode launch writes each new
token (position L - s_q + i) in the work item whose list range holds it:
its packed tile, or its protected row.  Restated here from that definition,
the rule must name exactly one work item per token, and that work item's
packed phase (a packed token) or protected phase (a protected token) must
read the token's position.
"""
import itertools

TILE = 32


def plan(L, sink, recent, split):
    """The key list and its work items, as the protected split planner and
    the decode launch lay them out."""
    has_packed = L - recent > sink
    pk0 = sink // TILE if has_packed else 0
    n_pk = -(-(L - recent) // TILE) - pk0 if has_packed else 0
    n_prot = sink + recent if has_packed else L
    n_list = n_pk + -(-n_prot // TILE)
    per = split // TILE if split else n_list
    items = [(u, min(u + per, n_list)) for u in range(0, n_list, per)]
    return pk0, n_pk, n_prot, items


def owner(L, sink, recent, items, pk0, n_pk, p):
    nsink, r0 = min(sink, L), max(sink, L - recent)
    prot = p < sink or p >= L - recent
    u = n_pk + (min(p, nsink) + max(0, p - r0)) // TILE if prot else p // TILE - pk0
    return [j for j, (u0, u1) in enumerate(items) if u0 <= u < u1], prot


def test_every_new_token_is_written_by_the_work_item_that_reads_it():
    n = 0
    for L, sink, recent, split, s_q in itertools.product(range(1, 400), [0, 1, 4, 40], [0, 1, 8, 16, 128],
                                                        [0, 32, 64, 96, 544], [1, 2]):
        if sink + recent < 1 or L < s_q:
            continue
        pk0, n_pk, n_prot, items = plan(L, sink, recent, split)
        nsink, r0 = min(sink, L), max(sink, L - recent)
        for i in range(s_q):
            p = L - s_q + i
            owners, prot = owner(L, sink, recent, items, pk0, n_pk, p)
            assert len(owners) == 1, (L, sink, recent, split, s_q, p, owners)
            u0, u1 = items[owners[0]]
            if prot:
                # the protected phase reads protected rows [vb, ve) of the list
                idx = min(p, nsink) + max(0, p - r0)
                vb, ve = TILE * (max(u0, n_pk) - n_pk), min(TILE * (u1 - n_pk), n_prot)
                assert vb <= idx < ve, (L, sink, recent, split, p)
            else:
                # the packed phase reads positions [tb, te)
                tb, te = TILE * (pk0 + u0), min(TILE * (pk0 + min(u1, n_pk)), L - recent)
                assert u0 < n_pk and tb <= p < te, (L, sink, recent, split, p)
            n += 1
    assert n > 100_000
