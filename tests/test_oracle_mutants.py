"""The pins must be strong enough to catch a plausible mistake anywhere in the
oracle.  Each case plants one mistake in a copy of lede_oracle.c (on the
CPU, in a temporary directory), builds it, and runs the pin checks against
that copy in a child process; the child must report a failure."""
import os
import subprocess
import sys
import textwrap

import pytest

from oracle.build import build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "lede_oracle.c")

# (name, text to replace, replacement, which occurrence (1-based))
MUTANTS = [
    ("rope_sign", "v[i] = x0 * c - x1 * s;", "v[i] = x0 * c + x1 * s;", 1),
    ("rope_freq", "pow(base, -2.0 * i / hd)", "pow(base, -1.0 * i / hd)", 1),
    ("attn_scale", "double scale = 1.0 / sqrt((double)hd);", "double scale = 1.0;", 1),
    ("gqa_map", "kvh = h / group", "kvh = h % nkv", 1),
    ("causal_excludes_self", "n = pos + 1;", "n = pos > 0 ? pos : 1;", 1),
    ("silu_dropped", "g[i] = act_round(M, z / (1.0 + exp(-z)) * up[i]);",
     "g[i] = act_round(M, z * up[i]);", 1),
    ("attn_residual_dropped", "for (size_t i = 0; i < (size_t)T * d; ++i) x[i] += y[i];",
     "for (size_t i = 0; i < (size_t)T * d; ++i) x[i] = y[i];", 1),
    ("ffn_residual_dropped", "for (size_t i = 0; i < (size_t)T * d; ++i) x[i] += y[i];",
     "for (size_t i = 0; i < (size_t)T * d; ++i) x[i] = y[i];", 2),
    ("norm_without_mean", "double inv = 1.0 / sqrt(ss / d + eps);", "double inv = 1.0 / sqrt(ss + eps);", 1),
    ("k_uses_wq", "matvec_rows(M, M->wk[l], kvd, d, u, T, k);", "matvec_rows(M, M->wq[l], kvd, d, u, T, k);", 1),
    ("gate_uses_up", "matvec_rows(M, M->wg[l], F, d, u, T, g);", "matvec_rows(M, M->wu[l], F, d, u, T, g);", 1),
    ("kv_not_rounded", "kc[i] = act_round(M, k[(size_t)t * kvd + i]);", "kc[i] = k[(size_t)t * kvd + i];", 1),
    ("attn_out_not_rounded", "o[i] = act_round(M, o[i]);", "o[i] = o[i];", 1),
    ("round_half_up", "nearbyint(m * 256.0)", "floor(m * 256.0 + 0.5)", 1),
    ("rope_wrong_position", "int pos = pos0 + t;\n      for (int h = 0; h < nq; ++h)",
     "int pos = pos0 + t + 1;\n      for (int h = 0; h < nq; ++h)", 1),
    ("head_skips_final_norm",
     "rmsnorm(M, hidden + (size_t)t * d, M->final_norm, d, M->eps, u + (size_t)t * d);",
     "memcpy(u + (size_t)t * d, hidden + (size_t)t * d, sizeof(double) * d);", 1),
    ("ffn_norm_uses_attn_gain", "rmsnorm(M, x + (size_t)t * d, M->ffn_norm[l]",
     "rmsnorm(M, x + (size_t)t * d, M->attn_norm[l]", 1),
]

CHILD = textwrap.dedent(r"""
    import sys
    sys.path.insert(0, {root!r})
    from tests.test_oracle_pins import (MICRO_F32, MICRO_BF16, MICRO_GQA, MICRO_GQA_BF16)
    import tests.test_oracle_pins as P
    from oracle import model as om
    L = om.lib({so!r})
    om._lib = L          # every pin below now runs against the mutant
    checks = [P.test_round_bf16_matches_torch_on_fp32_values, P.test_rope_closed_form_values,
              P.test_attend_matches_sdpa_and_special_cases, P.test_rmsnorm_matches_library_and_unit_rms]
    checks += [lambda m=m: P.test_decoder_matches_torch_bruteforce(m)
               for m in (MICRO_F32, MICRO_BF16, MICRO_GQA, MICRO_GQA_BF16)]
    # a non-trivial non-uniform gain, so that gain mix-ups are visible
    for c in checks:
        try:
            c()
        except Exception as e:
            print("CAUGHT", type(e).__name__)
            sys.exit(3)
    print("NOT CAUGHT")
""")


def _mutate(text, old, new, nth):
    idx = -1
    for _ in range(nth):
        idx = text.find(old, idx + 1)
        assert idx >= 0, "mutation anchor not found: %r" % old
    return text[:idx] + new + text[idx + len(old):]


@pytest.mark.parametrize("name,old,new,nth", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(tmp_path, name, old, new, nth):
    text = open(SRC).read()
    mutated = _mutate(text, old, new, nth)
    assert mutated != text
    src = tmp_path / ("mut_%s.c" % name)
    src.write_text(mutated)
    so = build(force=True, src=str(src), out=str(tmp_path / ("mut_%s.so" % name)))
    code = CHILD.format(root=ROOT, so=so)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert "NOT CAUGHT" not in r.stdout, "pins missed the planted mistake %s" % name
    assert r.returncode != 0
