"""The seeded input generator: determinism, slicing, distribution, shapes (CPU only)."""
import hashlib

import numpy as np
import pytest

import workloads as W


def test_philox_known_answers():
    # Known-answer vectors of Philox4x32-10 published with the Random123 library.
    assert W.philox4x32_10((0, 0, 0, 0), (0, 0)) == [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]
    assert W.philox4x32_10((0xFFFFFFFF,) * 4, (0xFFFFFFFF, 0xFFFFFFFF)) == [
        0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]
    assert W.philox4x32_10((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344),
                           (0xA4093822, 0x299F31D0)) == [0xD16CFE09, 0x94FDCCEB, 0x5001E420,
                                                         0x24126EA1]


def test_normal_distribution():
    x = W.normal_f32(123, 1, 2, 0, 1 << 20).astype(np.float64)
    assert abs(x.mean()) < 5e-3 and abs(x.std() - 1) < 5e-3
    assert abs((np.abs(x) > 2).mean() - 0.0455) < 2e-3


def test_slices_are_consistent():
    a = W.normal_bf16(7, 2, 3, 0, 10007)
    b = W.normal_bf16(7, 2, 3, 4093, 311)
    assert np.array_equal(a[4093:4093 + 311], b)
    wl = W.make_workload("tiny_extend")
    full = wl.k_rows(2, 0, int(wl.seq_lens[2]))
    assert np.array_equal(full[250:270], wl.k_rows(2, 250, 270))


@pytest.mark.parametrize("key", sorted(W.SPECS))
def test_workload_shapes(key):
    wl = W.make_workload(key)
    s = wl.spec
    assert wl.prefix_lens.shape == (s.num_tasks,) and wl.extend_lens.shape == (s.num_tasks,)
    final = wl.final_lens
    used = []
    for b in range(s.num_tasks):
        n = -(-int(final[b]) // 16)
        row = wl.block_table[b]
        assert (row[:n] >= 0).all() and (row[:n] < wl.num_pages).all()
        assert (row[n:] == -1).all()
        sp = 0 if wl.shared_lens is None else int(wl.shared_lens[wl.group_of(b)]) // 16
        used.extend(row[sp:n].tolist())  # a group's prompt pages are checked below
    if wl.shared_lens is not None:
        for g in range(len(wl.shared_lens)):
            s0, s1 = int(wl.group_start[g]), int(wl.group_start[g + 1])
            sp = int(wl.shared_lens[g]) // 16
            assert (wl.block_table[s0:s1, :sp] == wl.block_table[s0, :sp]).all()
            used.extend(wl.block_table[s0, :sp].tolist())
    assert len(used) == len(set(used)), "a physical page is shared by two tasks"
    if key == "tiny_extend":
        assert wl.prefix_lens.tolist() == [37, 100, 250, 511]
        assert wl.extend_lens.tolist() == [5, 17, 64, 128] and wl.num_pages == 128
    if key == "agent_resume_7b":
        assert wl.prefix_lens.min() >= 2048 and wl.prefix_lens.max() <= 16384
        assert wl.extend_lens.min() >= 64 and wl.extend_lens.max() <= 2048
    if key == "resumed_decode":
        ctx = wl.seq_lens
        assert ctx.min() >= 1024 and ctx.max() <= 32768 and (wl.extend_lens == 1).all()
        assert 5000 < np.median(ctx) < 7500
    if key == "multimodal_resume":
        assert wl.extend_lens.min() >= 1024 and wl.extend_lens.max() <= 4096
        frac = np.mean(np.concatenate(wl.outliers))
        assert 0.09 < frac < 0.11
    if key == "long_horizon":
        pref_pages = sum(-(-int(p) // 16) for p in wl.prefix_lens)
        assert abs(pref_pages / wl.num_pages - 0.9) < 1e-3
    if key == "multimodal_prune_resume":
        images, keep, img, text = s.prune
        assert (images, keep, img) == (10, 5, 1196)
        assert wl.prefix_lens.min() >= 512 and wl.prefix_lens.max() <= 2048
        # the pre-prune context holds ten screenshots and ten texts; the pruned sequence
        # lost exactly five screenshots and nothing else
        after = wl.stale_lens - wl.prefix_lens
        assert (after >= 10 * (img + text[1])).all() and (after <= 10 * (img + text[2])).all()
        assert ((wl.stale_lens - wl.seq_lens) == 5 * img).all()
        assert (wl.final_lens == wl.stale_lens).all()


def test_prune_rule_on_explicit_turns():
    """Sliding window (Appendix C): with ten screenshots in context the five oldest are
    dropped and every turn's text is kept, so the first changed position is the first
    screenshot, right after the prompt."""
    texts = [[3] * 10, [0] * 10, list(range(10))]
    wl = W.custom_prune_workload(8, 2, 64, [0, 16, 37], texts, image_tokens=16, seed=1)
    assert wl.prefix_lens.tolist() == [0, 16, 37]
    assert wl.stale_lens.tolist() == [0 + 160 + 30, 16 + 160, 37 + 160 + 45]
    assert wl.extend_lens.tolist() == [80 + 30, 80, 80 + 45]
    keep_all = W.custom_prune_workload(8, 2, 64, [20], [[1] * 10], keep=10, image_tokens=16)
    assert keep_all.extend_lens.tolist() == [0] and keep_all.stale_lens.tolist() == [190]


def test_stale_rows_are_their_own_stream():
    wl = W.make_workload(W.SPECS["multimodal_prune_resume"].shrunk(4, 16))
    b = 1
    p, s = int(wl.prefix_lens[b]), int(wl.stale_lens[b])
    old = wl.stale_rows("k", b, p, s)
    new = wl.k_rows(b, p, s)
    assert old.shape == new.shape and (old != new).mean() > 0.9
    assert np.array_equal(wl.stale_rows("k", b, p + 5, p + 9), old[5:9])
    assert not np.array_equal(wl.stale_rows("v", b, p, s), old)


def test_determinism_digest():
    a = W.make_workload("agent_resume_7b")
    b = W.make_workload("agent_resume_7b")
    assert a.lens_digest() == b.lens_digest()
    assert np.array_equal(a.block_table, b.block_table)
    h1 = hashlib.sha256(a.q_rows(5, 100, 140).tobytes()).hexdigest()
    h2 = hashlib.sha256(b.q_rows(5, 100, 140).tobytes()).hexdigest()
    assert h1 == h2


def test_group_workload_shares_prompt_values():
    """GRPO groups: every trajectory of a group holds the same K/V on the shared prompt
    positions (they are the same pages) and its own values after them; Q is per task."""
    wl = W.make_workload("grpo_group_decode")
    assert wl.group_start[0] == 0 and wl.group_start[-1] == wl.num_tasks
    assert (np.diff(wl.group_start) == wl.spec.group_size).all()
    assert (wl.shared_lens % 16 == 0).all() and (wl.shared_lens >= 2048 - 16).all()
    for g in (0, 17, 31):
        s0 = int(wl.group_start[g])
        sh = int(wl.shared_lens[g])
        assert (wl.seq_lens[s0:s0 + 8] > sh).all()
        a = wl.k_rows(s0, sh - 3, sh + 3)
        b = wl.k_rows(s0 + 5, sh - 3, sh + 3)
        assert (a[:3] == b[:3]).all() and not (a[3:] == b[3:]).all()
        va, vb = wl.v_rows(s0 + 1, 0, 20), wl.v_rows(s0 + 7, 0, 20)
        assert (va == vb).all()
        assert not (wl.q_rows(s0, 0, 4) == wl.q_rows(s0 + 1, 0, 4)).all()
