"""Plant plausible mistakes in copies of the CPU oracle and check that the
pins reject every one of them (CPU only; nothing here touches a GPU)."""
import os
import subprocess
import sys

import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle  # noqa: E402
import oracle_pins as P  # noqa: E402

SRC = os.path.join(os.path.dirname(oracle.__file__), "lmoracle.c")

# (name, text in lmoracle.c, replacement)
MUTANTS = [
    ("sample_low_word", "ids[i] = (int64_t)(uint64_t)(p >> 64);", "ids[i] = (int64_t)(uint64_t)p % V;"),
    ("sample_modulo_bias", "const unsigned __int128 p = (unsigned __int128)r[i] * (unsigned __int128)(uint64_t)V;",
     "const unsigned __int128 p = (unsigned __int128)(r[i] >> 1) * (unsigned __int128)(uint64_t)V;"),
    ("f16_ties_away", "if (rest > 0x1000u || (rest == 0x1000u && (h & 1u))) h += 1;",
     "if (rest >= 0x1000u) h += 1;"),
    ("f16_truncates", "if (rest > 0x1000u || (rest == 0x1000u && (h & 1u))) h += 1;", ""),
    ("f16_subnormal_shift", "const int s = 14 - e; /* bits dropped, 14..24 */",
     "const int s = 13 - e; /* bits dropped, 14..24 */"),
    ("f16_exponent_bias", "const int e = exp32 - 127 + 15;", "const int e = exp32 - 127 + 16;"),
    ("compress_scale_dropped", "const float t = x32 * scale;", "const float t = x32;"),
    ("decompress_scale_inverted", "const float g = f16_value(h[i]) * inv_scale;",
     "const float g = f16_value(h[i]) / inv_scale;"),
    ("ties_reversed", "if (x->k != y->k) return x->k < y->k ? -1 : 1;",
     "if (x->k != y->k) return x->k < y->k ? 1 : -1;"),
    ("last_token_dropped", "for (int64_t i = 0; i < K; ++i) {\n    if (i == 0",
     "for (int64_t i = 0; i < K - 1; ++i) {\n    if (i == 0"),
    ("offsets_off_by_one", "offsets[U] = (int32_t)i;", "offsets[U] = (int32_t)(i + 1);"),
    ("counts_not_accumulated", "counts[U - 1] += 1;", "counts[U - 1] = 1;"),
    ("inverse_by_sorted_position", "inverse[t[i].k] = (int32_t)(U - 1);",
     "inverse[i] = (int32_t)(U - 1);"),
    ("segsum_row_index_transposed",
     "for (int64_t d = 0; d < D; ++d) out[u * D + d] += grad_at(grad, gtype, ld, k, d);",
     "for (int64_t d = 0; d < D; ++d) out[u * D + d] += grad_at(grad, gtype, ld, u, d);"),
    ("bf16_widening_shift", "<< 16;\n  float f;", "<< 15;\n  float f;"),
    ("dense_overwrites", "dense[J[k] * D + d] += grad_at", "dense[J[k] * D + d] = grad_at"),
    ("lower_bound_off", "if (a[mid] < x) lo = mid + 1; else hi = mid;\n  }\n  return (lo < n",
     "if (a[mid] <= x) lo = mid + 1; else hi = mid;\n  }\n  return (lo < n"),
    ("expand_not_zero_filled", "memset(dst, 0, (size_t)(n_dst * D) * sizeof(double));\n  for (int64_t u = 0; u < n_src",
     "for (int64_t u = 0; u < n_src"),
    ("scatter_add_ignored", "if (add) dst[r * D + d] += src[u * D + d];",
     "if (add) dst[r * D + d] = src[u * D + d];"),
    ("sgd_sign", "p[i] -= lr * g[i];", "p[i] += lr * g[i];"),
    ("adam_bias_exponent", "double c1 = 1.0 - pow(b1, (double)t);",
     "double c1 = 1.0 - pow(b1, (double)(t + 1));"),
    ("adam_v_uncorrected", "double vhat = v[i] / c2;", "double vhat = v[i];"),
    ("adam_eps_inside_sqrt", "(sqrt(vhat) + eps)", "sqrt(vhat + eps)"),
    ("adam_decay_dropped", "+ wd * p[i]);", ");"),
    ("segsum_cols_shifted_column",
     "for (int64_t d = d0; d < d1; ++d) out[u * D + d] += grad_at(grad, gtype, ld, k, d);",
     "for (int64_t d = d0; d < d1; ++d) out[u * D + d] += grad_at(grad, gtype, ld, k, d - d0);"),
    ("segsum_cols_clears_every_column",
     "for (int64_t d = d0; d < d1; ++d) out[u * D + d] = 0.0;",
     "for (int64_t d = 0; d < D; ++d) out[u * D + d] = 0.0;"),
    ("select_skips_first_token", "for (int64_t k = 0; k < K; ++k) {\n    int64_t lo = 0, hi = nsel;",
     "for (int64_t k = 1; k < K; ++k) {\n    int64_t lo = 0, hi = nsel;"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_reject_mutant(tmp_path, name, old, new):
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation site for {name} not unique"
    src = tmp_path / "mutant.c"
    src.write_text(text.replace(old, new))
    so = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                    "-o", str(so), str(src), "-lm"], check=True)
    failed = []
    with oracle.loaded_from(str(so)):
        for check in P.ALL_CHECKS:
            try:
                check()
            except Exception as e:  # a pin failing, or the mutant crashing a check
                failed.append((check.__name__, type(e).__name__))
                break  # one rejection is enough
    assert failed, f"no pin caught mutant {name}"
