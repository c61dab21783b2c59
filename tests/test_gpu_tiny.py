"""Tiny-stack parity: libnova (through the C ABI) against the oracle on the same seeded inputs.

fp32 mode must reproduce the oracle's greedy ids exactly (the prefill's top-1/top-2 margin is
about 1e-4 of a 0.33-std logit, so only a near-fp32 path can); bf16 mode must stay within the
2e-2 relative bound with decode teacher-forced on the oracle's ids."""
import numpy as np
import pytest

from oracle import vlm
from tests import stage_cases as sc

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ref():
    return sc.oracle_tiny()


def test_tiny_fp32_exact_mode(gpu_lib, ref):
    out = sc.gpu_tiny(gpu_lib, gpu_lib.ACT_F32, ref)
    assert vlm.max_rel_err(out["vis"], ref["vis"]) < sc.TOL_F32
    ek, ev = sc.kv_errors(ref["kv_prefill"][0], ref["kv_prefill"][1], out["k_prefill"], out["v_prefill"])
    assert ek < sc.TOL_F32 and ev < sc.TOL_F32
    for t, (g, o) in enumerate(zip(out["logits"], ref["logits"])):
        assert vlm.max_rel_err(g, o) < sc.TOL_F32, f"step {t}"
    assert out["tokens"] == ref["tokens"]
    ek, ev = sc.kv_errors(ref["kv"].k, ref["kv"].v, out["k_final"], out["v_final"])
    assert ek < sc.TOL_F32 and ev < sc.TOL_F32


def test_tiny_bf16_teacher_forced(gpu_lib, ref):
    forced = ref["tokens"][:-1]
    out = sc.gpu_tiny(gpu_lib, gpu_lib.ACT_BF16, ref, forced=forced)
    assert vlm.max_rel_err(out["vis"], ref["vis"]) < sc.TOL_BF16
    ek, ev = sc.kv_errors(ref["kv_prefill"][0], ref["kv_prefill"][1], out["k_prefill"], out["v_prefill"])
    assert ek < sc.TOL_BF16 and ev < sc.TOL_BF16
    for t, (g, o) in enumerate(zip(out["logits"], ref["logits"])):
        assert vlm.max_rel_err(g, o) < sc.TOL_BF16, f"step {t}"
    # greedy ids agree wherever the oracle's top-1/top-2 margin exceeds the bf16 error of that step
    for t, (g, o) in enumerate(zip(out["logits"], ref["logits"])):
        top = np.sort(o)[::-1]
        err = np.abs(g - o).max()
        if top[0] - top[1] > 2 * err:
            assert int(np.argmax(g)) == int(np.argmax(o)), f"step {t}"


# A varied instruction fed step by step: with the oracle's own greedy ids the tiny stack repeats one
# token (its LM head favours it), which pins a single argmax.  Teacher-forced on seeded random ids,
# the oracle's per-step argmax moves over several tokens with top-1/top-2 margins of 0.01-0.18
# (step 0, the prefill, 1e-4), so every step's id is a separate check.
FORCED_SEED = 31


@pytest.fixture(scope="module")
def ref_forced():
    from paper_2509_21301_amd import synth
    forced = [int(t) for t in synth.text_ids(synth.TINY_DECODE_STEPS, synth.TINY_LLM.vocab, seed=FORCED_SEED)]
    return forced, sc.oracle_tiny(forced=forced)


def test_tiny_fp32_teacher_forced_varied_ids(gpu_lib, ref_forced):
    forced, ref = ref_forced
    assert len(set(ref["tokens"])) >= 4            # the check is not one repeated argmax
    out = sc.gpu_tiny(gpu_lib, gpu_lib.ACT_F32, ref, forced=forced)
    for t, (g, o) in enumerate(zip(out["logits"], ref["logits"])):
        assert vlm.max_rel_err(g, o) < sc.TOL_F32, f"step {t}"
    assert out["tokens"] == ref["tokens"]
    ek, ev = sc.kv_errors(ref["kv"].k, ref["kv"].v, out["k_final"], out["v_final"])
    assert ek < sc.TOL_F32 and ev < sc.TOL_F32


def test_tiny_bf16_teacher_forced_varied_ids(gpu_lib, ref_forced):
    forced, ref = ref_forced
    out = sc.gpu_tiny(gpu_lib, gpu_lib.ACT_BF16, ref, forced=forced)
    checked = 0
    for t, (g, o) in enumerate(zip(out["logits"], ref["logits"])):
        assert vlm.max_rel_err(g, o) < sc.TOL_BF16, f"step {t}"
        top = np.sort(o)[::-1]
        if top[0] - top[1] > 2 * np.abs(g - o).max():
            assert int(np.argmax(g)) == int(np.argmax(o)), f"step {t}"
            checked += 1
    assert checked >= 8
