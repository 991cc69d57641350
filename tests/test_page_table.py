"""Host page allocator and page tables of libjfkv.so (CPU only, no GPU calls).

Behaviour follows the paper's paging (Background, "Compact histories need
reusable storage": fixed pool, page table per request, page IDs returned on
completion), reference-counted shared prefixes with all-or-nothing
reservation (Sec. 3.3, eq. reservation) and recycling of zero-reference pages
after release (Algorithm 1).
"""
import numpy as np
import pytest

jfkv = pytest.importorskip("paper_2609_17475_amd.jfkv")


def test_identity_order_and_stats():
    pp = jfkv.PagePool(8, 256)
    s = pp.create()
    pp.reserve(s, 3 * 256 + 1)
    bt, lens = pp.export([s], 6)
    assert bt == [[0, 1, 2, 3, -1, -1]] and lens == [0]
    pp.set_length(s, 3 * 256 + 1)
    assert pp.export([s], 4)[1] == [769]
    assert pp.stats() == {"free": 4, "used": 4, "high_water": 4}


def test_shuffled_order_is_a_seeded_permutation():
    a, b = jfkv.PagePool(64, 256, 5), jfkv.PagePool(64, 256, 5)
    sa, sb = a.create(), b.create()
    a.reserve(sa, 64 * 256)
    b.reserve(sb, 64 * 256)
    ta = a.export([sa], 64)[0][0]
    assert ta == b.export([sb], 64)[0][0]
    assert sorted(ta) == list(range(64)) and ta != list(range(64))
    c = jfkv.PagePool(64, 256, 6)
    sc = c.create()
    c.reserve(sc, 64 * 256)
    assert c.export([sc], 64)[0][0] != ta


def test_reserve_is_all_or_nothing():
    pp = jfkv.PagePool(4, 64)
    s = pp.create()
    pp.reserve(s, 100)  # 2 pages
    with pytest.raises(jfkv.JfError) as e:
        pp.reserve(s, 64 * 5)
    assert e.value.status == jfkv.JF_ERR_NO_PAGES
    assert pp.info(s) == (2, 0)
    assert pp.stats()["free"] == 2
    pp.reserve(s, 256)
    assert pp.stats()["free"] == 0


def test_fork_shares_prefix_pages_and_release_recycles_lifo():
    pp = jfkv.PagePool(10, 64)
    a = pp.create()
    pp.reserve(a, 64 * 3)
    pp.set_length(a, 64 * 3)
    b = pp.fork(a, 128)
    assert pp.info(b) == (2, 128)
    bt, _ = pp.export([a, b], 4)
    assert bt[1][:2] == bt[0][:2]
    pp.reserve(b, 129)  # new own page
    bt, _ = pp.export([a, b], 4)
    assert bt[1][2] not in bt[0]
    assert pp.stats()["used"] == 4
    pp.release(a)  # shared pages survive, a's own page goes back
    assert pp.stats()["used"] == 3
    freed_last = bt[0][2]
    c = pp.create()
    pp.reserve(c, 1)
    assert pp.export([c], 1)[0][0][0] == freed_last  # last released, first reused
    pp.release(b)
    assert pp.stats()["used"] == 1
    with pytest.raises(jfkv.JfError) as e:
        pp.release(b)
    assert e.value.status == jfkv.JF_ERR_STATE


def test_append_into_shared_page_is_refused():
    pp = jfkv.PagePool(10, 64)
    a = pp.create()
    pp.reserve(a, 64 * 2)
    pp.set_length(a, 100)  # second page partially used
    b = pp.fork(a, 64)
    pp.set_length(b, 64)
    pp.reserve(b, 65)  # fine: new page
    with pytest.raises(jfkv.JfError) as e:
        pp.fork(a, 128)  # 128 > length 100
    assert e.value.status == jfkv.JF_ERR_INVALID
    pp.set_length(a, 128)
    d = pp.fork(a, 128)
    pp.set_length(d, 64)  # pretend d only used the first page: next write is shared
    with pytest.raises(jfkv.JfError) as e:
        pp.reserve(d, 65)
    assert e.value.status == jfkv.JF_ERR_STATE


def test_fork_requires_page_aligned_prefix():
    pp = jfkv.PagePool(4, 64)
    a = pp.create()
    pp.reserve(a, 128)
    pp.set_length(a, 128)
    with pytest.raises(jfkv.JfError) as e:
        pp.fork(a, 100)
    assert e.value.status == jfkv.JF_ERR_INVALID


def test_assign_explicit_pages():
    pp = jfkv.PagePool(8, 64)
    s = pp.create()
    pp.assign(s, [7, 6, 5])
    assert pp.export([s], 3)[0] == [[7, 6, 5]]
    t = pp.create()
    with pytest.raises(jfkv.JfError) as e:
        pp.assign(t, [1, 6])
    assert e.value.status == jfkv.JF_ERR_STATE
    assert pp.info(t) == (0, 0)
    with pytest.raises(jfkv.JfError):
        pp.assign(t, [2, 2])
    pp.reserve(t, 64 * 5)  # never hands out assigned pages
    got = pp.export([t], 5)[0][0]
    assert not set(got) & {5, 6, 7} and len(set(got)) == 5
    assert pp.stats() == {"free": 0, "used": 8, "high_water": 8}


def test_export_checks_capacity_and_handles():
    pp = jfkv.PagePool(8, 64)
    s = pp.create()
    pp.reserve(s, 64 * 3)
    with pytest.raises(jfkv.JfError):
        pp.export([s], 2)
    with pytest.raises(jfkv.JfError):
        pp.export([s + 5], 4)
    with pytest.raises(jfkv.JfError):
        pp.set_length(s, 64 * 3 + 1)


def test_random_operation_sequence_keeps_accounting_consistent():
    rng = np.random.default_rng(0)
    NP, P = 40, 64
    pp = jfkv.PagePool(NP, P, shuffle_seed=9)
    live = {}
    for _ in range(400):
        op = rng.integers(0, 4)
        if op == 0 or not live:
            s = pp.create()
            live[s] = 0
        elif op == 1:
            s = list(live)[rng.integers(0, len(live))]
            n = live[s] + int(rng.integers(1, 200))
            try:
                pp.reserve(s, n)
                pp.set_length(s, n)
                live[s] = n
            except jfkv.JfError as e:
                assert e.status in (jfkv.JF_ERR_NO_PAGES, jfkv.JF_ERR_STATE)
        elif op == 2:
            s = list(live)[rng.integers(0, len(live))]
            pre = (live[s] // P) * P
            f = pp.fork(s, pre)
            live[f] = pre
        else:
            s = list(live)[rng.integers(0, len(live))]
            pp.release(s)
            del live[s]
        tables, lens = pp.export(list(live), NP) if live else ([], [])
        refs = {}
        for t in tables:
            for p in t:
                if p >= 0:
                    refs[p] = refs.get(p, 0) + 1
        st = pp.stats()
        assert st["used"] == len(refs)
        assert st["free"] == NP - len(refs)
        assert st["high_water"] >= st["used"]
