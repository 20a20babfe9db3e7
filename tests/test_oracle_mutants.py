"""Mutation check of the oracle's pins (CPU only).

Each case plants one plausible mistake into a private copy of the oracle's C
source (a dropped term, a wrong sign, a transposed operand, a wrong loop
bound), compiles it into a temporary shared object and runs every pin against
it in a child process.  The pins must reject every mutant; a mutant that
crashes the child (an out-of-bounds index) counts as rejected too.
"""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "lora_oracle.c")

# (id, original text, mutated text) -- each original must occur exactly once.
MUTANTS = [
    ("u_transposed_A", "acc += X[t * K + k] * A[j * K + k];", "acc += X[t * K + k] * A[k * r + j];"),
    ("u_short_loop", "for (int64_t k = 0; k < K; ++k) acc += X[t * K + k] * A[j * K + k];",
     "for (int64_t k = 1; k < K; ++k) acc += X[t * K + k] * A[j * K + k];"),
    ("y_transposed_W", "base += X[t * K + k] * W[n * K + k];", "base += X[t * K + k] * W[k * N + n];"),
    ("y_short_loop", "for (int64_t k = 0; k < K; ++k) base +=", "for (int64_t k = 0; k + 1 < K; ++k) base +="),
    ("y_dropped_scale", "Y[i * N + n] = base + s * lora;", "Y[i * N + n] = base + lora;"),
    ("y_wrong_sign", "Y[i * N + n] = base + s * lora;", "Y[i * N + n] = base - s * lora;"),
    ("y_dropped_lora", "Y[i * N + n] = base + s * lora;", "Y[i * N + n] = base;"),
    ("y_transposed_B", "lora += U[t * r + j] * B[n * r + j];", "lora += U[t * r + j] * B[j * N + n];"),
    ("grad_u_unscaled", "dU[t * r + j] = s * acc;", "dU[t * r + j] = acc;"),
    ("grad_u_transposed_B", "acc += dY[t * N + n] * B[n * r + j];", "acc += dY[t * N + n] * B[j * N + n];"),
    ("dx_dropped_lora", "out[k] += lora;", "out[k] += 0.0 * lora;"),
    ("dx_wrong_row_of_W", "const double *wrow = W + n * K;", "const double *wrow = W + (N - 1 - n) * K;"),
    ("dx_transposed_A", "lora += dU[t * r + j] * A[j * K + k];", "lora += dU[t * r + j] * A[k * r + j];"),
    ("da_wrong_sign", "acc += dU[t * r + j] * X[t * K + k];", "acc -= dU[t * r + j] * X[t * K + k];"),
    ("da_first_token_only", "for (int64_t t = 0; t < T; ++t) acc += dU[t * r + j] * X[t * K + k];",
     "for (int64_t t = 0; t < 1; ++t) acc += dU[t * r + j] * X[t * K + k];"),
    ("db_unscaled", "dB[n * r + j] = s * acc;", "dB[n * r + j] = acc;"),
    ("db_transposed_U", "acc += dY[t * N + n] * U[t * r + j];", "acc += dY[t * N + n] * U[j * T + t];"),
    ("dq_nibbles_swapped", "q = (k % 2 == 0) ? (byte & 0x0F) : (byte >> 4);",
     "q = (k % 2 == 0) ? (byte >> 4) : (byte & 0x0F);"),
    ("dq_wrong_group", "const int64_t g = k / G;", "const int64_t g = k / (2 * G);"),
    ("dq_scale_offset_swapped", "W[n * K + k] = S[n * ngroups + g] * (double)q + Bo[n * ngroups + g];",
     "W[n * K + k] = Bo[n * ngroups + g] * (double)q + S[n * ngroups + g];"),
    ("dq_dropped_offset", "W[n * K + k] = S[n * ngroups + g] * (double)q + Bo[n * ngroups + g];",
     "W[n * K + k] = S[n * ngroups + g] * (double)q;"),
    ("dq_8bit_as_nibble", "q = Wq[n * row_bytes + k];", "q = Wq[n * row_bytes + k] & 0x0F;"),
    ("dq_wrong_byte", "const uint8_t byte = Wq[n * row_bytes + k / 2];",
     "const uint8_t byte = Wq[n * row_bytes + k / 2 + (k / 2 + 1 < row_bytes)];"),
    ("ce_target_gradient_dropped", "for (int64_t d = 0; d < D; ++d) out[d] -= wt[d];",
     "for (int64_t d = 0; d < D; ++d) out[d] -= 0.0 * wt[d];"),
    ("ce_wrong_target_logit", "loss[i] = lse - z[tpos[i]];", "loss[i] = lse - z[0];"),
    ("ce_log_missing", "const double lse = m + log(s);", "const double lse = m + s;"),
    ("ce_unnormalised_probability", "const double p = exp(z[j] - lse);", "const double p = exp(z[j] - m);"),
    ("ce_ignores_J", "for (int64_t d = 0; d < D; ++d) acc += H[t * D + d] * W[J[j] * D + d];",
     "for (int64_t d = 0; d < D; ++d) acc += H[t * D + d] * W[j * D + d];"),
    ("ce_wrong_row_of_H", "for (int64_t d = 0; d < D; ++d) acc += H[t * D + d] * W[J[j] * D + d];",
     "for (int64_t d = 0; d < D; ++d) acc += H[i * D + d] * W[J[j] * D + d];"),
    ("topk_ascending", "  if (a->c > b->c) return -1;\n  if (a->c < b->c) return 1;",
     "  if (a->c > b->c) return 1;\n  if (a->c < b->c) return -1;"),
    ("topk_unnormalised", "row[j].c = den > 0.0 ? dot / den : 0.0;", "row[j].c = dot;"),
    ("topk_row_norm_only", "const double den = norm[i] * norm[j];", "const double den = norm[i];"),
    ("topk_ties_larger_index_first", "return (a->j > b->j) - (a->j < b->j);",
     "return (a->j < b->j) - (a->j > b->j);"),
]

CHILD = textwrap.dedent("""
    import sys
    sys.path[:0] = [{root!r}, {tests!r}]
    import oracle, oracle_pins
    o = oracle.load({lib!r})
    failed = oracle_pins.run_all(o)
    print("FAILED_PINS", ",".join(failed))
    sys.exit(0 if failed else 3)
""")


@pytest.mark.parametrize("mid,orig,mut", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_reject_mutant(tmp_path, mid, orig, mut):
    src = open(SRC).read()
    assert src.count(orig) == 1, f"mutation anchor for {mid} not unique/found"
    msrc = tmp_path / "mutant.c"
    msrc.write_text(src.replace(orig, mut))
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-o", str(lib), str(msrc), "-lm"],
                   check=True)
    code = CHILD.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=str(lib))
    env = dict(os.environ, OMP_NUM_THREADS="1")
    p = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env,
                       timeout=300)
    # exit 0: at least one pin failed (mutant caught); a crash is also a catch.
    assert p.returncode != 3, f"mutant {mid} passed every pin:\n{p.stdout}\n{p.stderr}"
