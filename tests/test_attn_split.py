"""The persistent bf16 attention's equal-chunk split, checked on the host through
the library's own split arithmetic (fe_test_attn_split runs the helper the
kernel runs): for ragged batches every work item of every (sequence, column)
segment -- its prefix chunks, then one item for its cascade keys -- is taken
exactly once, partial slots stay below the slots the workspace holds, the
slots of a segment are 0..np-1 in item order, and the count its first piece
stores equals its number of pieces."""
import numpy as np
import pytest


@pytest.fixture(scope="module")
def fe():
    from paper_2509_20416_amd import fe as _fe
    _fe.lib()
    return _fe


def _check(fe, plens, ncols, nch_ld, pmax, waves):
    pieces = fe.fe_test_attn_split(plens, ncols, nch_ld, pmax, waves)
    B = len(plens)
    # prefix chunks (at most nch_ld - 1) plus the cascade-key item
    chunks = [min(-(-int(p) // 64), nch_ld - 1) + 1 if 0 <= p <= pmax else 1 for p in plens]
    seen = {}
    for w, b, col, ch0, n, slot, np_ in pieces:
        assert 0 <= b < B and 0 <= col < ncols and n >= 1
        assert 0 <= ch0 and ch0 + n <= chunks[b], (b, ch0, n, chunks[b])
        assert 0 <= slot < nch_ld, (slot, nch_ld)
        seg = seen.setdefault((b, col), {"cover": np.zeros(chunks[b], np.int32), "slots": [],
                                         "np": None, "waves": []})
        seg["cover"][ch0:ch0 + n] += 1
        seg["slots"].append((ch0, slot))
        seg["waves"].append(w)
        if ch0 == 0:
            assert np_ >= 1
            seg["np"] = np_
        else:
            assert np_ == 0
    assert len(seen) == B * ncols, "a segment got no piece"
    for (b, col), seg in seen.items():
        assert (seg["cover"] == 1).all(), (b, col, seg["cover"])
        slots = [s for _, s in sorted(seg["slots"])]
        assert slots == list(range(len(slots))), (b, col, slots)
        assert seg["np"] == len(slots), (b, col, seg["np"], len(slots))
        assert seg["waves"] == sorted(seg["waves"])          # chunk order follows wave order
    # the waves' ranges are contiguous and balanced: chunk counts differ by at most one
    per_wave = np.bincount(pieces[:, 0], weights=pieces[:, 4]).astype(int)
    assert per_wave.max() - per_wave.min() <= 1
    assert per_wave.sum() == sum(chunks) * ncols
    return pieces


@pytest.mark.parametrize("seed", range(12))
def test_split_covers_ragged_batches(fe, seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 257))
    pmax = int(rng.choice([64, 700, 8192]))
    plens = rng.integers(0, pmax + 1, B)
    ncols = int(rng.choice([1, 2, 8, 40]))
    nch_ld = -(-pmax // 64) + 1
    waves = int(rng.choice([1, 7, 1024, 4096]))
    _check(fe, plens, ncols, nch_ld, pmax, waves)


def test_split_batch32_workload(fe):
    """The batch-32 bench shape: P_b ~ U[256, 8192], 8 KV heads, 1024 resident waves."""
    from fe_synth import configs as C
    from fe_synth import make_prefix_lens
    plens = make_prefix_lens(C.LLAMA8B_BF16_B32, 0)
    _check(fe, plens, 8, -(-int(plens.max()) // 64) + 1, int(plens.max()), 1024)


def test_split_edge_cases(fe):
    _check(fe, [0], 1, 1, 0, 1024)                      # empty prefix: the cascade-key item alone
    _check(fe, [0] * 256, 8, 2, 64, 1024)
    _check(fe, [8192] * 256, 8, 129, 8192, 1024)        # the largest batch
    _check(fe, [1, 64, 65, 128, 129], 3, 4, 129, 2)
    # prefixes outside [0, pmax] count as empty (no cache row is read)
    pieces = _check(fe, [5000, 10, 99999], 2, 3, 128, 64)
    assert not ((pieces[:, 1] == 0) & (pieces[:, 3] > 0)).any()
