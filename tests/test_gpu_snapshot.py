"""GPU page-run snapshots (jf_kv_pack_pages / jf_kv_unpack_pages,
jf_snapshot_save / jf_snapshot_restore) against the oracle's pool bytes.

The expected snapshot of a layer is, by definition, the bytes of the
request's pages in logical order: for page table[i], its K codes, K (scale,
bias), V codes and V (scale, bias) runs for all KV heads, taken from the
oracle's pool (built from the same rows, byte-equal to the device pool).
Checks: packed pages equal those bytes (a page outside the pool packs as
zeros; a host buffer is refused before any launch); the file is a valid
safetensors file (read back with the safetensors package, a loader that
executes nothing) whose tensors equal them; staging buffers from two pages
to all of them; a partial last page; n_pos = 0;
restoring into pages of a differently shuffled pool reproduces every byte,
and decode over the restored request equals decode over the original
bitwise; a failed save leaves an existing file untouched."""
import os

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from gpu_cases import POISON, build, decode_gpu, log  # noqa: E402

from paper_2609_17475_amd import jfkv  # noqa: E402

DEV = "cuda"


def expected_pages(host_pool, lay, table, n_pages):
    """Oracle pool bytes of pages table[0 .. n_pages-1]: [n_pages][page_bytes]."""
    P, hkv, d, G = lay.page_size, lay.num_kv_heads, lay.head_dim, lay.group_size
    cb = hkv * P * d // 2
    mb = hkv * P * (d // G) * 4
    runs = [host_pool.k_codes.view(np.uint8).reshape(-1, cb),
            host_pool.k_meta.view(np.uint8).reshape(-1, mb),
            host_pool.v_codes.view(np.uint8).reshape(-1, cb),
            host_pool.v_meta.view(np.uint8).reshape(-1, mb)]
    out = []
    for i in range(n_pages):
        p = int(table[i])
        if 0 <= p < lay.num_pages:
            out.append(np.concatenate([r[p] for r in runs]))
        else:
            out.append(np.zeros(2 * (cb + mb), np.uint8))
    return np.stack(out) if out else np.zeros((0, 2 * (cb + mb)), np.uint8)


def layers(n, P=64, hkv=2, d=128, G=64, L=700, seed=0):
    """n layers of one request: same page table, different rows per layer."""
    return [build(P=P, hkv=hkv, d=d, G=G, hq=4 * hkv, lens=(L,), seed=seed + 31 * i,
                  shuffle_seed=5) for i in range(n)]


def staging(n_bytes):
    return torch.empty(n_bytes, dtype=torch.uint8).pin_memory()


def test_pack_unpack_match_pool_bytes():
    log("snapshot pack/unpack")
    (case,) = layers(1, L=1000)
    lay = case.lay
    pb = jfkv.kv_page_bytes(lay)
    table = case.tables[0].copy()
    n_pages = -(-1000 // lay.page_size)
    table[3] = -1  # a page outside the pool packs as zeros
    t_dev = torch.from_numpy(table).to(DEV)
    buf = torch.full((n_pages * pb,), POISON, dtype=torch.uint8, device=DEV)
    jfkv.jf_kv_pack_pages(case.gpu, t_dev, 0, n_pages, buf)
    torch.cuda.synchronize()
    got = buf.cpu().numpy().reshape(n_pages, pb)
    assert np.array_equal(got, expected_pages(case.host, lay, table, n_pages))
    # unpack into a poisoned pool through another mapping, pack again
    other = jfkv.KVPool(lay, device=DEV, fill=POISON)
    perm = np.random.default_rng(3).permutation(lay.num_pages)[:n_pages].astype(np.int32)
    p_dev = torch.from_numpy(perm).to(DEV)
    jfkv.jf_kv_unpack_pages(other, p_dev, 0, n_pages, buf)
    back = torch.empty_like(buf)
    jfkv.jf_kv_pack_pages(other, p_dev, 0, n_pages, back)
    torch.cuda.synchronize()
    assert torch.equal(back.cpu(), buf.cpu())
    # host memory is refused before any launch (kernels never dereference it)
    with pytest.raises(jfkv.JfError) as e:
        jfkv.jf_kv_pack_pages(case.gpu, t_dev, 0, n_pages, staging(n_pages * pb))
    assert e.value.status == jfkv.JF_ERR_INVALID


@pytest.mark.parametrize("stage_pages,L", [(2, 700), (5, 700), (64, 700), (3, 64 * 11 + 5),
                                          (2, 0)])
def test_save_matches_pool_bytes_and_restores(tmp_path, stage_pages, L):
    from safetensors.numpy import load_file
    log("snapshot save/restore staging=%d pages L=%d" % (stage_pages, L))
    cases = layers(3, L=max(L, 1))
    lay = cases[0].lay
    pb = jfkv.kv_page_bytes(lay)
    P = lay.page_size
    n_pages = -(-L // P)
    table = cases[0].tables[0]
    t_dev = torch.from_numpy(table).to(DEV)
    st = staging(stage_pages * pb)
    sd = torch.empty(stage_pages * pb, dtype=torch.uint8, device=DEV)
    path = str(tmp_path / "prefix.safetensors")
    jfkv.snapshot_save(path, [c.gpu for c in cases], t_dev, table, L, sd, st)
    assert os.path.exists(path) and not os.path.exists(path + ".tmp")
    data = load_file(path)
    assert sorted(data) == ["layer0", "layer1", "layer2"]
    for i, c in enumerate(cases):
        assert data["layer%d" % i].shape == (n_pages, pb)
        assert np.array_equal(data["layer%d" % i], expected_pages(c.host, lay, table, n_pages))
    # restore into a fresh, poisoned pool through a differently shuffled table
    pp = jfkv.PagePool(lay.num_pages, P, shuffle_seed=99)
    s = pp.create()
    pp.reserve(s, max(L, 1))
    table2 = np.array(pp.export([s], table.shape[0])[0][0], np.int32)
    pools2 = [jfkv.KVPool(lay, device=DEV, fill=POISON) for _ in cases]
    n_pos = jfkv.snapshot_restore(path, pools2, torch.from_numpy(table2).to(DEV), table2, sd, st)
    assert n_pos == L
    for p2, c in zip(pools2, cases):
        buf = torch.empty(max(n_pages, 1) * pb, dtype=torch.uint8, device=DEV)
        jfkv.jf_kv_pack_pages(p2, torch.from_numpy(table2).to(DEV), 0, n_pages, buf)
        torch.cuda.synchronize()
        got = buf.cpu().numpy()[:n_pages * pb].reshape(n_pages, pb)
        assert np.array_equal(got, expected_pages(c.host, lay, table, n_pages))
    if L > 0:  # the restored request decodes bitwise as the original
        q = (np.random.default_rng(7).standard_normal((1, cases[0].hq, lay.head_dim))
             / np.sqrt(lay.head_dim)).astype(np.float16)
        for p2, c in zip(pools2, cases):
            a = decode_gpu(c, q)
            c2 = type(c)(**{**c.__dict__, "gpu": p2, "tables": table2[None]})
            b = decode_gpu(c2, q)
            assert np.array_equal(a, b)


def test_failed_save_leaves_existing_file(tmp_path):
    (case,) = layers(1)
    lay = case.lay
    pb = jfkv.kv_page_bytes(lay)
    path = tmp_path / "keep.safetensors"
    path.write_bytes(b"previous contents")
    bad = case.tables[0].copy()
    bad[1] = lay.num_pages + 5
    sd = torch.empty(2 * pb, dtype=torch.uint8, device=DEV)
    with pytest.raises(jfkv.JfError) as e:
        jfkv.snapshot_save(str(path), [case.gpu], torch.from_numpy(bad).to(DEV), bad, 700, sd,
                           staging(2 * pb))
    assert e.value.status == jfkv.JF_ERR_INVALID
    assert path.read_bytes() == b"previous contents"
    with pytest.raises(jfkv.JfError) as e:  # a directory that does not exist
        jfkv.snapshot_save(str(tmp_path / "no" / "such.safetensors"), [case.gpu],
                           torch.from_numpy(case.tables[0]).to(DEV), case.tables[0], 700, sd,
                           staging(2 * pb))
    assert e.value.status == jfkv.JF_ERR_IO
