"""Home map of an allocation and the local / remote read kernel on the device,
through the C ABI.

The read kernel is checked bit-exactly: the XOR of every 16-byte word it reads
must equal the XOR of the same chunks computed on the host, for every list
mode, partial XCD sets and three chunk sizes.  The home map is checked against
its own verification lines (random lines timed separately, whose measured home
must match the map) with the partition hash the interleave probe measures on
the same device.  Bandwidths and latency tiers are printed, not pinned.
"""
import numpy as np
import pytest

import paper_2609_24270_amd as asym

pytestmark = pytest.mark.gpu

GRP = [0, 0, 0, 0, 1, 1, 1, 1]
PAGE = 2 << 20


@pytest.fixture(scope="module")
def dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    asym.load_library()
    return torch.device("cuda:0")


def _aligned(dev, nbytes, fill_seed=None):
    import torch
    raw = torch.empty(nbytes + PAGE, dtype=torch.uint8, device=dev)
    shift = (-raw.data_ptr()) % PAGE
    buf = raw[shift: shift + nbytes]
    if fill_seed is not None:
        g = torch.Generator(device=dev).manual_seed(fill_seed)
        buf.view(torch.int32).copy_(torch.randint(-2**31, 2**31 - 1, (nbytes // 4,), generator=g,
                                                  device=dev, dtype=torch.int32))
    return raw, buf


def _host_xor(host_words, chunk_log2, chunks):
    """XOR of the 16-byte words (as 4 uint32) of the listed chunks."""
    per = (1 << chunk_log2) // 16
    w = host_words.reshape(-1, per, 4)
    if len(chunks) == 0:
        return np.zeros(4, dtype=np.uint32)
    return np.bitwise_xor.reduce(w[np.asarray(chunks, dtype=np.int64)].reshape(-1, 4), axis=0)


@pytest.mark.parametrize("chunk_log2", [12, 13, 16])
def test_read_kernel_checksum_is_exact(dev, chunk_log2):
    import torch
    nbytes = 64 << 20
    raw, buf = _aligned(dev, nbytes, fill_seed=chunk_log2)
    torch.cuda.synchronize()
    words = buf.view(torch.int32).cpu().numpy().view(np.uint32)
    n_chunks = nbytes >> chunk_log2
    g = np.random.default_rng(chunk_log2)
    home = g.choice([-1, 0, 1], size=n_chunks, p=[0.1, 0.45, 0.45]).astype(np.int8)
    for mode in (asym.CHUNKS_ALL, asym.CHUNKS_LOCAL, asym.CHUNKS_REMOTE):
        for xm in (0, 0x0F, 0x81):
            chunks, off = asym.chunk_lists(home, 8, GRP, mode, xm)
            ms, ck = asym.chunk_read_bw(buf.data_ptr(), nbytes, chunk_log2, chunks, off, iters=2)
            want = _host_xor(words, chunk_log2, chunks)
            assert ck.tolist() == want.tolist(), (mode, xm)
            assert ms > 0
            # few workers per XCD (each reads the list of the XCD it runs on)
            for w in (1, 3):
                _, ck = asym.chunk_read_bw(buf.data_ptr(), nbytes, chunk_log2, chunks, off, iters=1,
                                           workers_per_xcd=w)
                assert ck.tolist() == want.tolist(), (mode, xm, w)


def test_read_kernel_rejects(dev):
    raw, buf = _aligned(dev, 4 << 20)
    chunks = np.array([0, 1, 512], dtype=np.uint32)       # 512 is beyond 4 MiB of 8 KiB chunks
    off = np.array([0, 3, 3, 3, 3, 3, 3, 3, 3], dtype=np.int32)
    with pytest.raises(asym.AsymError):
        asym.chunk_read_bw(buf.data_ptr(), 4 << 20, 13, chunks, off)
    ok = np.array([0, 1, 2], dtype=np.uint32)
    with pytest.raises(asym.AsymError):
        asym.chunk_read_bw(buf.data_ptr(), 4 << 20, 11, ok, off)
    with pytest.raises(asym.AsymError):
        asym.chunk_read_bw(buf.data_ptr(), 4 << 20, 13, ok, off[:5])   # not the device's XCD count
    with pytest.raises(asym.AsymError):
        asym.chunk_read_bw(buf.data_ptr() + 8, 4 << 20, 13, ok, off)
    bad = off.copy()
    bad[2] = 1
    with pytest.raises(asym.AsymError):
        asym.chunk_read_bw(buf.data_ptr(), 4 << 20, 13, ok, bad)       # decreasing offsets


def test_home_map_agrees_with_its_verification_lines(dev):
    r, *_ = asym.interleave_probe(0, n_bases=64, lo_bit=7, hi_bit=24, n_pairs=2, passes=2)
    assert r["n_groups"] == 2, r["group_of_xcd"]
    chunk_log2 = max(12, r["lowest_bit"])
    raw, buf = _aligned(dev, 1 << 30)
    info, homes = asym.home_map(buf.data_ptr(), 1 << 30, r["hash_mask"], chunk_log2,
                                group_of_xcd=r["group_of_xcd"], passes=2, n_verify=2048, seed=3)
    print({k: info[k] for k in ("n_pages", "unclassified_pages", "chunk_share", "verify_classified",
                                "verify_agree", "local_cycles", "remote_cycles")},
          "hash", hex(r["hash_mask"]), "chunk", 1 << chunk_log2, flush=True)
    assert info["n_chunks"] == homes.shape[0] == (1 << 30) >> chunk_log2
    assert info["verify_classified"] >= 0.9 * 2048
    assert info["verify_agree"] >= 0.98 * info["verify_classified"]
    assert info["unclassified_pages"] <= info["n_pages"] // 20
    assert info["local_cycles"] < info["remote_cycles"]
    # reading with the map: local, remote and all, printed
    out = {}
    for name, mode in (("all", asym.CHUNKS_ALL), ("local", asym.CHUNKS_LOCAL), ("remote", asym.CHUNKS_REMOTE)):
        chunks, off = asym.chunk_lists(homes, 8, info["group_of_xcd"], mode)
        ms, _ = asym.chunk_read_bw(buf.data_ptr(), 1 << 30, chunk_log2, chunks, off, iters=5)
        out[name] = round(len(chunks) * (1 << chunk_log2) / (ms * 1e-3) / 1e9, 1)
    print("GB/s on 1 GiB", out, flush=True)
