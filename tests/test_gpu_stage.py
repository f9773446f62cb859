"""D2D staging guard and gather on the GPU vs the CPU oracle (bit-exact)."""
import numpy as np
import pytest

from oracle import stage as stage_oracle
import paper_2607_17181_amd as tsa

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _words_dev(bits):
    return torch.from_numpy(stage_oracle.bits_to_words(bits).view(np.int32)).cuda()


def _layout(rng, n_chunks, chunk, gap):
    rows, so = [], 4096
    for i in range(n_chunks):
        size = chunk if i % 7 else chunk // 2 + 16   # ragged sizes, multiples of 16
        rows.append((so, i * chunk, size))
        so += size + gap
    return np.array(rows, dtype=np.int64), so + 4096, n_chunks * chunk


@pytest.mark.parametrize("n_chunks,chunk,page", [(45, 8192, 4096), (200, 65536, 16384), (7, 1 << 20, 65536)])
def test_mark_dirty_and_gather_bit_exact(n_chunks, chunk, page):
    rng = np.random.default_rng(n_chunks)
    chunks, stage_bytes, wbytes = _layout(rng, n_chunks, chunk, gap=4096)
    host = rng.integers(0, 256, wbytes, dtype=np.uint8)
    staging = rng.integers(0, 256, stage_bytes, dtype=np.uint8)
    num_pages = stage_bytes // page + 1
    used = rng.random(num_pages) < 0.1
    staged = rng.random(n_chunks) < 0.8
    weights0 = rng.integers(0, 256, wbytes, dtype=np.uint8)
    # a malformed entry (unaligned weight offset) is skipped
    chunks[3, 1] += 8
    ch = torch.from_numpy(chunks).cuda()
    dirty_d = torch.zeros((n_chunks + 31) // 32, dtype=torch.int32, device="cuda")
    tsa.stage_mark_dirty(ch, _words_dev(used), num_pages, page, dirty_d)
    dirty_ref = stage_oracle.mark_dirty(chunks, used, page)
    assert np.array_equal(dirty_d.cpu().numpy().view(np.uint32), stage_oracle.bits_to_words(dirty_ref))
    hw = torch.empty(wbytes, dtype=torch.uint8, pin_memory=True)
    hw.copy_(torch.from_numpy(host))
    wd = torch.from_numpy(weights0).cuda()
    tsa.stage_gather(ch, _words_dev(staged), dirty_d, torch.from_numpy(staging).cuda(), hw, wd)
    ref = stage_oracle.gather(chunks, staged, dirty_ref, staging, host, weights0)
    assert np.array_equal(wd.cpu().numpy(), ref)


def test_guard_recovers_host_weights_after_kv_allocation():
    rng = np.random.default_rng(9)
    chunks, stage_bytes, wbytes = _layout(rng, 64, 32768, gap=0)
    host = rng.integers(0, 256, wbytes, dtype=np.uint8)
    staging = np.zeros(stage_bytes, dtype=np.uint8)
    for so, wo, nb in chunks:
        staging[so:so + nb] = host[wo:wo + nb]
    page = 4096
    num_pages = stage_bytes // page + 1
    used = np.zeros(num_pages, bool)
    used[rng.choice(num_pages, 40, replace=False)] = True
    st = torch.from_numpy(staging).cuda()
    for p in np.nonzero(used)[0]:          # the KV allocator writes rows into used pages
        st[p * page:(p + 1) * page] = torch.randint(0, 256, (page,), dtype=torch.uint8).cuda()
    ch = torch.from_numpy(chunks).cuda()
    dirty = torch.zeros(2, dtype=torch.int32, device="cuda")
    tsa.stage_mark_dirty(ch, _words_dev(used), num_pages, page, dirty)
    hw = torch.empty(wbytes, dtype=torch.uint8, pin_memory=True)
    hw.copy_(torch.from_numpy(host))
    wd = torch.zeros(wbytes, dtype=torch.uint8, device="cuda")
    tsa.stage_gather(ch, _words_dev(np.ones(64, bool)), dirty, st, hw, wd)
    got = wd.cpu().numpy()
    covered = np.zeros(wbytes, bool)
    for _, wo, nb in chunks:
        covered[wo:wo + nb] = True
    assert np.array_equal(got[covered], host[covered])   # every chunk holds the host bytes
    assert not got[~covered].any()                        # bytes outside chunks untouched
