"""The pins must catch plausible mistakes in the oracle.

Each case plants one mistake in a private copy of oracle.c (dropped bias, sign
error, transposed weight operand, missing ReLU or clamp, off-by-one in a loop,
fp32 accumulation, wrong bias index), builds it on the CPU, and checks that the
battery of independent pins rejects it.  The committed oracle must pass the
same battery.
"""

import json
import math
import os
import shutil

import numpy as np
import pytest

import oracle
from tests import brute
from workloads import Layer, dense_to_csr, integer_shadow, make_config, tiny_random

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

_ACC_BLOCK = """        for (int64_t t = 0; t < cur_len; ++t) {
            const int32_t i = cur_col[t];
            const double y = (double)cur_val[t];
            for (int64_t e = W->row_ptr[i]; e < W->row_ptr[i + 1]; ++e) {
                acc[W->col[e]] += y * (double)W->val[e];
                if (job->bias_mode && y != 0.0) touched[W->col[e]] = 1;
            }
        }"""

_TRANSPOSED = """        for (int64_t t = 0; t < cur_len; ++t) {
            const int32_t i = cur_col[t];
            const double y = (double)cur_val[t];
            for (int64_t j2 = 0; j2 < n; ++j2)
                for (int64_t e = W->row_ptr[j2]; e < W->row_ptr[j2 + 1]; ++e)
                    if (W->col[e] == i) {
                        acc[j2] += y * (double)W->val[e];
                        if (job->bias_mode && y != 0.0) touched[j2] = 1;
                    }
        }"""

MUTANTS = {
    "drop_bias": ("double z = acc[j] + (double)W->bias[j];", "double z = acc[j];"),
    "sign": ("acc[W->col[e]] += y * (double)W->val[e];", "acc[W->col[e]] -= y * (double)W->val[e];"),
    "transposed_W": (_ACC_BLOCK, _TRANSPOSED),
    "no_relu": ("if (z < 0.0) z = 0.0;", ""),
    "no_clamp": ("if (z > job->ymax) z = job->ymax;", ""),
    "skip_last_weight": ("e < W->row_ptr[i + 1]; ++e) {\n                acc",
                         "e + 1 < W->row_ptr[i + 1]; ++e) {\n                acc"),
    "skip_first_input": ("for (int64_t t = 0; t < cur_len; ++t) {\n            const int32_t i",
                         "for (int64_t t = 1; t < cur_len; ++t) {\n            const int32_t i"),
    "fp32_accumulate": ("acc[W->col[e]] += y * (double)W->val[e];",
                        "acc[W->col[e]] = (float)(acc[W->col[e]] + (float)(y * (double)W->val[e]));"),
    "bias_index": ("(double)W->bias[j];\n            if (z < 0.0)", "(double)W->bias[0];\n            if (z < 0.0)"),
    "keep_zero": ("if (f != 0.0f) {", "if (f != 0.0f || j == 0) {"),
    "pattern_bias_everywhere": ("if (job->bias_mode && !touched[j]) continue;", ""),
    "pattern_touch_zero_inputs": ("if (job->bias_mode && y != 0.0) touched[W->col[e]] = 1;",
                                  "if (job->bias_mode) touched[W->col[e]] = 1;"),
    "pattern_never_touch": ("if (job->bias_mode && y != 0.0) touched[W->col[e]] = 1;", ""),
    "scale_signed": ("s[W->col[e]] += fabs(p);", "s[W->col[e]] += p;"),
    "scale_doubled": ("s[W->col[e]] += fabs(p);", "s[W->col[e]] += 2.0 * fabs(p);"),
    "scale_no_bias": ("s[j] += fabs((double)W->bias[j]);", ""),
    "preact_no_bias": ("z[j] += (double)W->bias[j];", ""),
}


def battery(lib):
    """Independent pins; returns the names of those that fail."""
    failed = []
    g = json.load(open(os.path.join(GOLDEN, "hand_example.json")))
    W = np.array(g["W"], np.float32)
    rp, c, v = dense_to_csr(W)
    lay = [Layer(rp, c, v, np.array(g["b"], np.float32))] * 2
    y0 = dense_to_csr(np.array(g["Y0"], np.float32))
    try:
        out = oracle.forward(3, lay, math.inf, y0, lib=lib)
        if not np.array_equal(oracle.csr_to_dense(out, 3), np.array(g["Y2"], np.float32)):
            failed.append("hand")
        out = oracle.forward(3, lay, 8.0, y0, lib=lib)
        if not np.array_equal(oracle.csr_to_dense(out, 3), np.array(g["ymax8_Y2"], np.float32)):
            failed.append("hand_clamp")
        for seed in (1, 2):
            p = tiny_random(seed, 17, 3, 4, w_density=0.4, y_density=0.8)
            got = oracle.forward(17, p.layers, math.inf, p.y0_csr, lib=lib)
            if not np.all(got[2] != 0):
                failed.append("no_stored_zeros")
            want = brute.dense_forward(oracle.csr_to_dense(p.y0_csr, 17), [l.to_dense(17) for l in p.layers],
                                       [l.bias for l in p.layers])
            if oracle.csr_to_dense(got, 17).tobytes() != want.tobytes():
                failed.append(f"brute{seed}")
        q = integer_shadow(make_config(3, n=256, L=2, batch=6))
        Yi = oracle.csr_to_dense(q.y0_csr, 256).astype(np.int64)
        for l in q.layers:
            Yi = np.clip(Yi @ l.to_dense(256).astype(np.int64) + l.bias.astype(np.int64), 0, 1000)
        got = oracle.forward(256, q.layers, q.ymax, q.y0_csr, lib=lib)
        if not np.array_equal(oracle.csr_to_dense(got, 256), Yi.astype(np.float32)):
            failed.append("integer_shadow")
        want = dense_to_csr(Yi.astype(np.float32))  # canonical CSR of the exact answer
        if not (np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])):
            failed.append("integer_shadow_pattern")
        # bias on the structural pattern (reading B): the hand example, and the pattern-semantics listing
        # on random inputs with positive biases and explicit zeros in Y_0
        out = oracle.forward(3, lay, math.inf, y0, lib=lib, bias_mode=1)
        if not np.array_equal(oracle.csr_to_dense(out, 3), np.array(g["pattern_bias"]["Y2"], np.float32)):
            failed.append("hand_pattern")
        # pre-activation and its condition scale s = |Y||W| + |b|: hand-worked values, then the exact
        # integer case against a library matmul of the absolute values
        z, s = oracle.preact(3, lay[0], y0, lib=lib)
        if not (np.array_equal(z, np.array(g["Y0W_plus_b"], np.float64))
                and np.array_equal(s, np.array(g["S_scale"], np.float64))):
            failed.append("hand_preact")
        z, s = oracle.preact(256, q.layers[0], q.y0_csr, lib=lib)
        Yq = oracle.csr_to_dense(q.y0_csr, 256).astype(np.int64)
        Wq = q.layers[0].to_dense(256).astype(np.int64)
        bq = q.layers[0].bias.astype(np.int64)
        if not (np.array_equal(z, (Yq @ Wq + bq).astype(np.float64))
                and np.array_equal(s, (np.abs(Yq) @ np.abs(Wq) + np.abs(bq)).astype(np.float64))):
            failed.append("integer_preact")
        for seed in (3, 4):
            p = tiny_random(seed, 19, 3, 5, w_density=0.15, y_density=0.3, bias_lo=-0.2, bias_hi=0.6,
                            explicit_zeros=True)
            y0d = oracle.csr_to_dense(p.y0_csr, 19)
            got = oracle.forward(19, p.layers, math.inf, p.y0_csr, lib=lib, bias_mode=1)
            want = brute.fig4_forward_pattern(y0d, [l.entries() for l in p.layers], [l.bias for l in p.layers])
            if oracle.csr_to_dense(got, 19).tobytes() != want.tobytes():
                failed.append(f"pattern{seed}")
    except ValueError:
        failed.append("error")
    return failed


def test_committed_oracle_passes_battery():
    assert battery(oracle.load()) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    src = open(os.path.join(os.path.dirname(oracle.__file__), "oracle.c")).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    lib = oracle.load(oracle.build(str(tmp_path / "libmutant.so"), str(path)))
    assert battery(lib), f"mutant {name} passed every pin"
