"""CPU oracle for the TQ4 codec and for decode attention over TQ4 vectors.

TEST INFRASTRUCTURE ONLY: like the rest of ``oracle/``, only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it.  Plain numpy, float64 except where the paper fixes a precision (the
centroids are float32, the stored norm is an fp16 rounding of a float32 norm).

Paper: "JustFit: Just-in-Time State Management for Local LLM Serving".
  * encoding and reconstruction: Sec. 3.1, eq. (codec): the vector is divided
    by its norm and rotated by H_d S / sqrt(d) (H_d the unnormalised Hadamard
    matrix, S a diagonal of random signs); each rotated coordinate becomes the
    index of one of 16 shared centroids; reconstruction multiplies the stored
    fp16 norm by S H_d / sqrt(d) applied to the centroid values;
  * storage: Background, eq. for the TQ4 payload (128 packed bytes plus a
    two-byte norm per 256-element vector) and Appendix A, Table codec (32 u32
    words of eight indices each, an fp16 norm computed from an fp32 norm);
  * codebook: Appendix A, Table codec (16 float32 centroids for the density
    proportional to (1 - x^2)^((d - 3) / 2), built on a 32,768-point grid of
    [-1 + 1e-6, 1 - 1e-6] from a quantile start with at most 100 centroid
    updates, stopping once no centroid moves by 1e-6 or more);
  * random signs: Appendix A, Table codec (NumPy default_rng with seed
    seed + 7919 d, K seed 0 and V seed 1);
  * quantization: Appendix A, Table codec (thresholds at the midpoints of
    adjacent centroids, a coordinate passes a threshold only if strictly
    greater);
  * attention over the reconstructed vectors: Sec. 3.1 (eq. groupattention),
    the plain softmax definition, heads independent.

Readings where the paper leaves a detail open (each listed with its reason in
the design notes):
  * "quantile initialization": centroid i starts at the (i + 1/2)/16 quantile
    of the grid density (the centres of 16 equal-mass cells);
  * a centroid update sets every centroid to the density-weighted mean of the
    grid points whose index under the current thresholds is i (a cell with no
    weight keeps its centroid); the stop test compares each update with the
    centroids before it;
  * "sampling +-1": rng.choice([-1, 1], size=d), d draws in coordinate order
    (parity unpinned: nothing outside this reading fixes which +-1 sequence
    the seed yields; a kernel takes the signs as an input, so its parity
    does not depend on it);
  * the norm is the float64 Euclidean norm rounded to float32, then to fp16
    (round to nearest even at both steps); encoding divides by the float32
    norm, reconstruction multiplies by the fp16 one;
  * index order in a word: element 8w + k of a vector sits in bits 4k..4k+3 of
    word w (the same little-endian order as the affine codes);
  * a zero vector encodes with norm 0 and every rotated coordinate taken as
    0 (its indices are those of a coordinate equal to 0), and reconstructs
    as 0.
"""
from __future__ import annotations

import numpy as np

GRID_POINTS = 32768
GRID_EPS = 1e-6
MAX_UPDATES = 100
STOP_CHANGE = 1e-6
SIGN_SEED_STRIDE = 7919
K_SEED, V_SEED = 0, 1
LEVELS = 16


def density(x: np.ndarray, d: int) -> np.ndarray:
    """Unnormalised density (1 - x^2)^((d - 3)/2) of one coordinate of a
    uniform point on the unit sphere in d dimensions (Table codec)."""
    return np.power(1.0 - x * x, (d - 3) / 2.0)


def codebook(d: int, grid: int = GRID_POINTS, eps: float = GRID_EPS,
             max_updates: int = MAX_UPDATES, stop: float = STOP_CHANGE):
    """The 16 shared centroids for head dimension d, ascending, float32
    (Table codec: grid, quantile start, Lloyd updates, stop rule).

    Returns (centroids float32 [16], number of updates made)."""
    xs = np.linspace(-1.0 + eps, 1.0 - eps, grid)
    w = density(xs, d)
    cdf = np.cumsum(w) / np.sum(w)
    # quantile start: the grid point where the cumulative mass first reaches
    # the centre of each of 16 equal-mass cells
    targets = (np.arange(LEVELS) + 0.5) / LEVELS
    c = xs[np.searchsorted(cdf, targets)].astype(np.float64)
    updates = 0
    for _ in range(max_updates):
        t = 0.5 * (c[:-1] + c[1:])
        cell = np.searchsorted(t, xs, side="left")  # number of thresholds strictly below x
        new = c.copy()
        for i in range(LEVELS):
            m = cell == i
            wm = w[m].sum()
            if wm > 0:
                new[i] = (w[m] * xs[m]).sum() / wm
        change = np.max(np.abs(new - c))
        c = new
        updates += 1
        if change < stop:
            break
    return c.astype(np.float32), updates


def signs(d: int, seed: int) -> np.ndarray:
    """The random-sign diagonal S as float64 +-1 [d] (Table codec)."""
    rng = np.random.default_rng(seed + d * SIGN_SEED_STRIDE)
    return rng.choice(np.array([-1.0, 1.0]), size=d)


def hadamard(d: int) -> np.ndarray:
    """Unnormalised Sylvester Hadamard matrix H_d (entries +-1, d a power of
    two), built by repeated Kronecker products with [[1, 1], [1, -1]]."""
    if d < 1 or d & (d - 1):
        raise ValueError("d must be a power of two")
    h = np.ones((1, 1))
    base = np.array([[1.0, 1.0], [1.0, -1.0]])
    while h.shape[0] < d:
        h = np.kron(h, base)
    return h


def rotation(d: int, s: np.ndarray) -> np.ndarray:
    """R = H_d S / sqrt(d), the encoder's rotation (eq. codec)."""
    return hadamard(d) * s[None, :] / np.sqrt(d)


def thresholds(c: np.ndarray) -> np.ndarray:
    """Midpoints of adjacent centroids, float64 (exact for float32 inputs)."""
    c = c.astype(np.float64)
    return 0.5 * (c[:-1] + c[1:])


def norm_f32(x: np.ndarray) -> np.ndarray:
    """Euclidean norm of each row (float64 sum of squares), rounded to float32."""
    x = np.asarray(x, np.float64)
    return np.sqrt(np.sum(x * x, axis=-1)).astype(np.float32)


def encode(x: np.ndarray, s: np.ndarray, c: np.ndarray):
    """Encode rows of x [n][d] (eq. codec, Table codec).

    Returns (indices uint8 [n][d] in 0..15, fp16 norms [n], rotated unit
    vectors y float64 [n][d] (for tests))."""
    x = np.asarray(x, np.float64)
    n, d = x.shape
    rho = norm_f32(x).astype(np.float64)
    safe = np.where(rho > 0, rho, 1.0)
    y = (x / safe[:, None]) @ rotation(d, s).T
    y[rho == 0] = 0.0
    return quantize(y, c), rho.astype(np.float32).astype(np.float16), y


def quantize(y: np.ndarray, c: np.ndarray) -> np.ndarray:
    """Index of each rotated coordinate: the number of midpoint thresholds it
    strictly exceeds (Table codec), uint8 in 0..15."""
    idx = np.zeros(np.shape(y), np.uint8)
    for t in thresholds(c):
        idx += (np.asarray(y) > t).astype(np.uint8)  # a coordinate on a threshold stays below it
    return idx


def pack(idx: np.ndarray) -> np.ndarray:
    """Indices [n][d] -> u32 words [n][d/8], element 8w + k at bits 4k of word w."""
    idx = np.asarray(idx, np.uint32)
    n, d = idx.shape
    g = idx.reshape(n, d // 8, 8)
    words = np.zeros((n, d // 8), np.uint32)
    for k in range(8):
        words |= g[:, :, k] << np.uint32(4 * k)
    return words


def unpack(words: np.ndarray) -> np.ndarray:
    """u32 words [n][d/8] -> indices uint8 [n][d] (inverse of pack)."""
    words = np.asarray(words, np.uint32)
    n, nw = words.shape
    out = np.zeros((n, nw, 8), np.uint8)
    for k in range(8):
        out[:, :, k] = ((words >> np.uint32(4 * k)) & np.uint32(15)).astype(np.uint8)
    return out.reshape(n, nw * 8)


def reconstruct(idx: np.ndarray, norm16: np.ndarray, s: np.ndarray, c: np.ndarray) -> np.ndarray:
    """x_hat = rho_hat * S H_d c[z] / sqrt(d), float64 [n][d] (eq. codec)."""
    idx = np.asarray(idx)
    d = idx.shape[1]
    vals = c.astype(np.float64)[idx]
    return norm16.astype(np.float64)[:, None] * (vals @ rotation(d, s))


def vector_bytes(d: int) -> int:
    """Stored bytes per vector: d/2 packed index bytes and one fp16 norm
    (Background, eq. for the TQ4 payload)."""
    return d // 2 + 2


def gather(words_pool: np.ndarray, norm_pool: np.ndarray, table: np.ndarray, L: int):
    """Logical rows 0..L-1 of a paged TQ4 pool through a page table.

    words_pool u32 [NP][Hkv][P][d/8], norm_pool fp16 [NP][Hkv][P]; position t
    lives in page table[t // P], slot t % P (Background, page table).
    Returns (words [L][Hkv][d/8], norms [L][Hkv])."""
    P = words_pool.shape[2]
    t = np.arange(L)
    pages = np.asarray(table)[t // P]
    slots = t % P
    return words_pool[pages, :, slots], norm_pool[pages, :, slots]


def decode_attention(q: np.ndarray, k_words: np.ndarray, k_norm: np.ndarray,
                     v_words: np.ndarray, v_norm: np.ndarray, s_k: np.ndarray,
                     s_v: np.ndarray, c: np.ndarray, scale: float) -> np.ndarray:
    """Softmax attention of one request's query heads q [Hq][d] over L
    positions of TQ4 K/V in logical order (k_words [L][Hkv][d/8], k_norm
    [L][Hkv], same for V), query head h reading KV head h // (Hq / Hkv).
    Every vector is reconstructed by eq. (codec), then the plain definition
    runs in float64 (Sec. 3.1, eq. groupattention).  Returns float64 [Hq][d]."""
    q = np.asarray(q, np.float64)
    Hq, d = q.shape
    L, Hkv = k_norm.shape
    gq = Hq // Hkv
    out = np.zeros((Hq, d))
    for kv in range(Hkv):
        kh = reconstruct(unpack(k_words[:, kv]), k_norm[:, kv], s_k, c)
        vh = reconstruct(unpack(v_words[:, kv]), v_norm[:, kv], s_v, c)
        for h in range(kv * gq, (kv + 1) * gq):
            logits = scale * (kh @ q[h])
            p = np.exp(logits - logits.max())
            out[h] = (p @ vh) / p.sum()
    return out
