"""Pins of the D2D-staging oracle (CPU): byte-level brute force, the bitmap
packing, and the guard's defining property -- whatever the KV allocator wrote
into the staging region, the assembled weights equal the host copy as long
as the clean staged chunks were staged correctly."""
import numpy as np

from oracle import stage


def _layout(rng, n_chunks=12, chunk=256, gap=64):
    """Chunks staged back to back (with gaps) in a staging region."""
    rows, so = [], 32
    for i in range(n_chunks):
        rows.append((so, i * chunk, chunk))
        so += chunk + gap
    return np.array(rows, dtype=np.int64), so + 64, n_chunks * chunk


def test_mark_dirty_matches_byte_overlap():
    rng = np.random.default_rng(0)
    chunks, stage_bytes, _ = _layout(rng)
    page = 48
    used = rng.random(stage_bytes // page + 1) < 0.15
    d = stage.mark_dirty(chunks, used, page)
    for i, (so, _, nb) in enumerate(chunks):
        overlap = any(used[b // page] for b in range(so, so + nb) if b // page < len(used))
        assert d[i] == overlap


def test_gather_matches_byte_loop():
    rng = np.random.default_rng(1)
    chunks, stage_bytes, wbytes = _layout(rng)
    staging = rng.integers(0, 256, stage_bytes, dtype=np.uint8)
    host = rng.integers(0, 256, wbytes, dtype=np.uint8)
    weights = rng.integers(0, 256, wbytes, dtype=np.uint8)
    staged = rng.random(len(chunks)) < 0.7
    dirty = rng.random(len(chunks)) < 0.3
    out = stage.gather(chunks, staged, dirty, staging, host, weights)
    ref = weights.copy()
    for i, (so, wo, nb) in enumerate(chunks):
        for b in range(nb):
            ref[wo + b] = staging[so + b] if (staged[i] and not dirty[i]) else host[wo + b]
    assert np.array_equal(out, ref)


def test_guard_recovers_host_weights_whatever_kv_wrote():
    rng = np.random.default_rng(2)
    chunks, stage_bytes, wbytes = _layout(rng, n_chunks=20)
    host = rng.integers(0, 256, wbytes, dtype=np.uint8)
    staging = np.zeros(stage_bytes, dtype=np.uint8)
    for so, wo, nb in chunks:                      # correct staging
        staging[so:so + nb] = host[wo:wo + nb]
    page = 64
    used = rng.random(stage_bytes // page + 1) < 0.2
    for p in np.nonzero(used)[0]:                  # KV rows overwrite used pages
        staging[p * page:(p + 1) * page] = rng.integers(0, 256, page, dtype=np.uint8)
    dirty = stage.mark_dirty(chunks, used, page)
    assert dirty.any() and not dirty.all()
    out = stage.gather(chunks, np.ones(len(chunks), bool), dirty, staging, host,
                       np.zeros(wbytes, np.uint8))
    assert np.array_equal(out, host)
    # without the guard the corrupted bytes would have been copied
    bad = stage.gather(chunks, np.ones(len(chunks), bool), np.zeros(len(chunks), bool), staging,
                       host, np.zeros(wbytes, np.uint8))
    assert not np.array_equal(bad, host)


def test_bits_to_words():
    bits = np.zeros(70, bool)
    bits[[0, 31, 32, 69]] = True
    w = stage.bits_to_words(bits)
    assert list(w) == [0x80000001, 0x00000001, 0x20]
