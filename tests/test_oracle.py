"""The oracle against its pins (CPU only).  See oracle_pins.py for what each pin is."""
import os
import subprocess

import numpy as np
import pytest

import oracle
import oracle_pins as pins

WORKLOADS = pins.shrunk_workloads()
IDS = [wl.spec.key for wl in WORKLOADS]


def test_golden_closed_forms():
    pins.pin_golden()


@pytest.mark.parametrize("wl", WORKLOADS, ids=IDS)
def test_matches_torch_sdpa(wl):
    pins.pin_sdpa(wl)


def test_uniform_weights_and_causal_bound():
    pins.pin_uniform()


def test_constant_values_weights_sum_to_one():
    pins.pin_constant_v()


def test_single_key():
    pins.pin_one_key()


@pytest.mark.parametrize("wl", WORKLOADS[:2] + WORKLOADS[4:], ids=IDS[:2] + IDS[4:])
def test_page_permutation_invariance(wl):
    pins.pin_permutation(wl)


@pytest.mark.parametrize("wl", WORKLOADS[:2], ids=IDS[:2])
def test_gqa_replication(wl):
    pins.pin_gqa_replica(wl)


@pytest.mark.parametrize("wl", WORKLOADS, ids=IDS)
def test_append_placement(wl):
    pins.pin_append(wl)


def test_extend_equals_prefill_rows():
    """Resume over a retained prefix == rows P.. of the full prefill (fp64)."""
    wl = WORKLOADS[1]
    kp, vp = pins.oracle_pools_for(wl)
    q_ext = wl.packed("q", wl.extend_ranges())
    q_full = wl.packed("q", wl.full_ranges())
    ext, ext_lse = oracle.extend(q_ext, kp, vp, wl.block_table, wl.prefix_lens, wl.extend_lens,
                                 wl.spec.num_q_heads, wl.sm_scale)
    full, full_lse = oracle.prefill(q_full, kp, vp, wl.block_table, wl.seq_lens,
                                    wl.spec.num_q_heads, wl.sm_scale)
    row_e, row_f = 0, 0
    for b in range(wl.num_tasks):
        p, e = int(wl.prefix_lens[b]), int(wl.extend_lens[b])
        np.testing.assert_allclose(ext[row_e:row_e + e], full[row_f + p:row_f + p + e], atol=1e-12)
        np.testing.assert_allclose(ext_lse[row_e:row_e + e], full_lse[row_f + p:row_f + p + e],
                                   atol=1e-12)
        row_e += e
        row_f += p + e


def test_bad_page_is_an_error():
    kp, vp = oracle.new_pools(4, 1, 64)
    bt = np.array([[4]], np.int32)  # out of range
    z = np.zeros((1, 1, 64), np.uint16)
    with pytest.raises(ValueError):
        oracle.kv_append(z, z, kp, vp, bt, np.array([0], np.int32), np.array([1], np.int32))
    with pytest.raises(ValueError):
        oracle.decode(np.zeros((1, 1, 64), np.uint16), kp, vp, bt, np.array([1], np.int32), 1, 0.1)


# ---- planted mistakes: each broken oracle must fail at least one pin -----------------
MUTANTS = {
    "dropped_scale": ("s[p] = scale * dot;", "s[p] = dot;"),
    "causal_off_by_one": ("int64_t t = (int64_t)prefix_lens[b] + (row - indptr[b]);",
                          "int64_t t = (int64_t)prefix_lens[b] + (row - indptr[b]) + 1;"),
    "gqa_modulo_map": ("int g = h / group;", "int g = h % hkv;"),
    "v_read_from_k_pool": ("s[p] * bf16_bits_to_double(v_pool[", "s[p] * bf16_bits_to_double(k_pool["),
    "v_read_transposed": (
        "bf16_bits_to_double(v_pool[slot_index(page, g, slot, i, hkv, d)]);",
        "bf16_bits_to_double(v_pool[(((size_t)page * (size_t)hkv + (size_t)g) * (size_t)d + "
        "(size_t)i) * ORACLE_PAGE + (size_t)slot]);"),
    "softmax_sign": ("s[p] = exp(s[p] - m);", "s[p] = exp(m - s[p]);"),
    "lse_without_max": ("= m + log(z);", "= log(z);"),
    "unnormalized_output": ("o[i] /= z;", "o[i] /= 1.0;"),
    "slot_index_shift": ("int slot = (int)(p % ORACLE_PAGE);\n      double dot",
                         "int slot = (int)((p + 1) % ORACLE_PAGE);\n      double dot"),
    "append_row_index": ("size_t src = ((size_t)row *", "size_t src = ((size_t)j *"),
    "append_v_transposed": (
        "v_pool[slot_index(page, g, slot, i, hkv, d)] = v_new[src];",
        "v_pool[(((size_t)page * (size_t)hkv + (size_t)g) * (size_t)d + (size_t)i) * ORACLE_PAGE + "
        "(size_t)slot] = v_new[src];"),
}


def _run_pins(lib):
    failures = []
    checks = [
        ("golden", lambda: pins.pin_golden(lib)),
        ("uniform", lambda: pins.pin_uniform(lib)),
        ("constant_v", lambda: pins.pin_constant_v(lib)),
        ("one_key", lambda: pins.pin_one_key(lib)),
        ("sdpa", lambda: pins.pin_sdpa(WORKLOADS[0], lib)),
        ("append", lambda: pins.pin_append(WORKLOADS[0], lib)),
    ]
    for name, fn in checks:
        try:
            fn()
        except (AssertionError, ValueError):
            failures.append(name)
    return failures


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(oracle.SOURCE).read()
    assert src.count(old) >= 1, "mutation target not found: %r" % old
    path = tmp_path / ("oracle_%s.c" % name)
    path.write_text(src.replace(old, new))
    lib_path = str(tmp_path / ("liboracle_%s.so" % name))
    oracle.build(force=True, source=str(path), out=lib_path)
    failures = _run_pins(oracle.load(lib_path))
    assert failures, "mutant %s passed every pin" % name


def test_unmutated_oracle_passes_the_mutation_checks():
    assert _run_pins(oracle.load()) == []
