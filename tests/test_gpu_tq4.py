"""GPU TQ4 encode-and-append against the TQ4 oracle.

Every written slot holds the oracle's indices and fp16 norm; every other pool
byte keeps its poison fill.  Both sides decide an index by comparing a
rotated coordinate with a threshold, the kernel after an fp32 Walsh-Hadamard
transform, the oracle after an fp64 rotation: the two values differ by at
most ~5.4 fp32 unit roundoffs of the unit vector (the butterfly partial sums
after k of the 8 stages are at most 2^(k/2) |x|, plus the norm and the
division), so an index may differ, by one, only where the oracle's
coordinate lies within 1e-6 of that threshold; there both indices are
correct.  A norm may differ by one fp16 step only where the exact norm lies
within 1e-6 (relative) of the midpoint between the two.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from gpu_cases import log  # noqa: E402

from oracle import tq4  # noqa: E402
from paper_2609_17475_amd import jfkv  # noqa: E402

D = 256
POISON = 0xA5
BAND = 1e-6
_CB = {}


def codebook():
    if "c" not in _CB:
        _CB["c"] = tq4.codebook(D)[0]
    return _CB["c"]


def tables(rng, lens, starts, P, NP, holes=()):
    need = [-(-(st + n) // P) for n, st in zip(lens, starts)]
    max_pages = max(need)
    perm = rng.permutation(NP).astype(np.int32)
    t = np.full((len(lens), max_pages), -1, np.int32)
    off = 0
    for b, k in enumerate(need):
        t[b, :k] = perm[off:off + k]
        off += k
    assert off <= NP
    for b, p in holes:
        t[b, p] = -1
    return t


def encode_gpu(lay, x, signs, lens, starts, table, c=None):
    pool = jfkv.TQ4Pool(lay, fill=POISON)
    dev = torch.device("cuda:0")
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32, device=dev)
    st = torch.tensor(starts, dtype=torch.int32, device=dev)
    jfkv.jf_tq4_encode_append(pool, torch.from_numpy(x).to(dev),
                              torch.from_numpy(signs.astype(np.float32)).to(dev),
                              torch.from_numpy(codebook() if c is None else c).to(dev), cu, st,
                              torch.from_numpy(table).to(dev))
    torch.cuda.synchronize()
    return (pool.words.cpu().numpy().view(np.uint32), pool.norms.cpu().numpy())


def slots_of(lens, starts, table, P, rows=None):
    """(row, page, slot) of every written row (rows outside the table skipped)."""
    out = []
    r = 0
    for b, (n, s) in enumerate(zip(lens, starts)):
        for i in range(n):
            pos = s + i
            if rows is None or r in rows:
                lp = pos // P
                if 0 <= lp < table.shape[1] and table[b, lp] >= 0:
                    out.append((r, int(table[b, lp]), pos % P))
            r += 1
    return out


def check_vectors(x_rows, w_gpu, n_gpu, signs, c=None):
    """Compare the kernel's words and norms for vectors x_rows [m][D] with
    the oracle (codebook c, default the format's); returns the number of band
    cases."""
    c = codebook() if c is None else c
    idx, n16, y = tq4.encode(x_rows, signs, c)
    g_idx = tq4.unpack(w_gpu)
    diff = g_idx.astype(np.int32) - idx.astype(np.int32)
    bad = np.argwhere(diff != 0)
    t = tq4.thresholds(c)
    for i, j in bad:
        lo = min(idx[i, j], g_idx[i, j])
        assert abs(int(diff[i, j])) == 1, (i, j, idx[i, j], g_idx[i, j])
        assert abs(y[i, j] - t[lo]) < BAND, (i, j, y[i, j], t[lo])
    nb = np.argwhere(n16.view(np.uint16) != n_gpu.view(np.uint16))
    rho = np.sqrt(np.sum(np.asarray(x_rows, np.float64) ** 2, axis=1))
    for (i,) in nb:
        a, b = float(n16[i]), float(n_gpu[i])
        assert abs(int(n16.view(np.uint16)[i]) - int(n_gpu.view(np.uint16)[i])) == 1, (i, a, b)
        assert abs(rho[i] - 0.5 * (a + b)) <= 1e-6 * rho[i], (i, rho[i], a, b)
    return len(bad) + len(nb)


def run_case(P, hkv, lens, starts, NP, seed, x=None, signs_seed=tq4.K_SEED, holes=()):
    log("tq4 encode P=%d hkv=%d lens=%s starts=%s NP=%d seed=%d" % (P, hkv, lens, starts, NP,
                                                                    seed))
    rng = np.random.default_rng(seed)
    total = sum(lens)
    if x is None:
        x = rng.standard_normal((total, hkv, D)).astype(np.float16)
    table = tables(rng, lens, starts, P, NP, holes)
    lay = jfkv.layout(P, hkv, D, 64, NP)
    signs = tq4.signs(D, signs_seed)
    w, n = encode_gpu(lay, x, signs, lens, starts, table)
    written = np.zeros((NP, hkv, P), bool)
    sl = slots_of(lens, starts, table, P)
    rows = np.array([r for r, _, _ in sl], np.int64)
    pages = np.array([p for _, p, _ in sl], np.int64)
    slots = np.array([s for _, _, s in sl], np.int64)
    band = 0
    for kv in range(hkv):
        written[pages, kv, slots] = True
        band += check_vectors(x[rows, kv].astype(np.float64), w[pages, kv, slots],
                              n[pages, kv, slots], signs)
    # everything else keeps its poison bytes
    assert np.all(w[~written] == 0xA5A5A5A5)
    assert np.all(n.view(np.uint16)[~written] == 0xA5A5)
    log("  %d vectors, %d band cases" % (len(sl) * hkv, band))
    assert band <= max(4, len(sl) * hkv * D // 20000)
    return band


def test_single_request_several_pages():
    run_case(256, 4, (700,), (0,), 6, 1)


def test_ragged_batch_shuffled_pages():
    run_case(64, 2, (100, 1, 257), (30, 0, 64), 16, 2, signs_seed=tq4.V_SEED)


def test_rows_outside_the_table_are_skipped():
    # request 0: positions 0..299 with its second page missing (-1);
    # request 1: starts past its table's last page (nothing written)
    P, NP = 64, 12
    lens, starts = (300, 40), (0, 0)
    rng = np.random.default_rng(3)
    t = tables(rng, lens, starts, P, NP, holes=[(0, 1)])
    x = rng.standard_normal((340, 3, D)).astype(np.float16)
    lay = jfkv.layout(P, 3, D, 64, NP)
    signs = tq4.signs(D, 0)
    w, n = encode_gpu(lay, x, signs, lens, (0, t.shape[1] * P), t)
    sl = slots_of(lens, (0, t.shape[1] * P), t, P)
    assert len(sl) == 300 - 64
    written = np.zeros((NP, 3, P), bool)
    for r, p, s in sl:
        written[p, :, s] = True
    assert np.all(w[~written] == 0xA5A5A5A5)
    rows = np.array([r for r, _, _ in sl])
    pages = np.array([p for _, p, _ in sl])
    slots = np.array([s for _, _, s in sl])
    for kv in range(3):
        check_vectors(x[rows, kv].astype(np.float64), w[pages, kv, slots], n[pages, kv, slots],
                      signs)


def test_edge_vectors():
    rng = np.random.default_rng(4)
    n = 12
    x = rng.standard_normal((n, 2, D)).astype(np.float16)
    x[0] = 0.0                                   # zero vector
    x[1] = 0.0; x[1, :, 17] = 3.0                # one spike
    x[2] = np.float16(65504.0)                   # fp16 maximum everywhere
    x[2, :, ::3] = np.float16(-65504.0)
    x[3] = np.float16(2.0 ** -24)                # smallest subnormal everywhere
    x[4] = (rng.standard_normal((2, D)) * 2.0 ** -20).astype(np.float16)  # subnormal range
    x[5] = x[6] = x[7]                           # identical vectors
    x[8] = 1.0                                   # constant vector
    x[9] = np.float16(-0.0)                      # negative zeros
    run_case(32, 2, (n,), (5,), 2, 5, x=x)


def test_full_bulk_sampled():
    # 262,143 rows x 4 KV heads into 1,024 shuffled pages of 256 (the TQ4
    # geometry of the paper's full-attention layers); 4,096 sampled rows
    # against the oracle, every slot of the window written
    P, hkv, NP, L = 256, 4, 1032, 262143
    log("tq4 encode bulk L=%d" % L)
    rng = np.random.default_rng(6)
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(6)
    x = torch.randn((L, hkv, D), generator=g, device=dev, dtype=torch.float32).half()
    table = tables(rng, (L,), (0,), P, NP)
    lay = jfkv.layout(P, hkv, D, 64, NP)
    signs = tq4.signs(D, 0)
    pool = jfkv.TQ4Pool(lay, fill=POISON)
    jfkv.jf_tq4_encode_append(pool, x, torch.from_numpy(signs.astype(np.float32)).to(dev),
                              torch.from_numpy(codebook()).to(dev),
                              torch.tensor([0, L], dtype=torch.int32, device=dev),
                              torch.tensor([0], dtype=torch.int32, device=dev),
                              torch.from_numpy(table).to(dev))
    torch.cuda.synchronize()
    w = pool.words.cpu().numpy().view(np.uint32)
    nrm = pool.norms.cpu().numpy()
    used = table[0]
    # norms: every slot of the window written (a Gaussian row has norm > 0),
    # the one slot past it and the spare pages untouched
    nu = nrm.view(np.uint16)
    pos = np.arange(L)
    assert np.all(nu[used[pos // P], :, pos % P] != 0xA5A5)
    assert np.all(nu[used[L // P], :, L % P] == 0xA5A5)
    spare = np.setdiff1d(np.arange(NP), used)
    assert np.all(w[spare] == 0xA5A5A5A5)
    rows = np.sort(rng.choice(L, 4096, replace=False))
    xs = x[torch.from_numpy(rows).to(dev)].float().cpu().numpy().astype(np.float64)
    band = 0
    for kv in range(hkv):
        band += check_vectors(xs[:, kv], w[used[rows // P], kv, rows % P],
                              nrm[used[rows // P], kv, rows % P], signs)
    log("  band cases %d" % band)


@pytest.mark.parametrize("kind", ["clustered", "uniform"])
def test_other_codebooks(kind):
    """Codebooks other than the format's: one whose two middle thresholds lie
    within one bucket of the kernel's index table (the kernel falls back to a
    binary search), and uniform levels (the table path with other
    thresholds).  Indices and norms match the oracle with the same
    codebook."""
    log("tq4 encode, %s codebook" % kind)
    c = codebook().astype(np.float32).copy()
    if kind == "clustered":
        c[8] = np.float32(c[7] + 1e-4)
        c[9] = np.float32(c[8] + 1e-4)
    else:
        c = np.linspace(-0.2, 0.2, 16).astype(np.float32)
    rng = np.random.default_rng(11)
    P, hkv, NP = 64, 3, 8
    lens, starts = (200, 77), (0, 10)
    t = tables(rng, lens, starts, P, NP)
    x = rng.standard_normal((sum(lens), hkv, D)).astype(np.float16)
    signs = tq4.signs(D, 0)
    lay = jfkv.layout(P, hkv, D, 64, NP)
    w, n = encode_gpu(lay, x, signs, lens, starts, t, c=c)
    sl = slots_of(lens, starts, t, P)
    rows = np.array([r for r, _, _ in sl])
    pages = np.array([p for _, p, _ in sl])
    slots = np.array([q for _, _, q in sl])
    for kv in range(hkv):
        check_vectors(x[rows, kv].astype(np.float64), w[pages, kv, slots], n[pages, kv, slots],
                      signs, c=c)
