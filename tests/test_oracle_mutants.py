"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake (a dropped term, a wrong sign, index or bound, a
transposed operand) in a temporary copy of the oracle's C source, builds it,
and runs the pin tests against that build in a subprocess: they must fail.
Everything happens on the CPU; the real oracle is untouched.
"""
import os
import subprocess
import sys

import pytest

from oracle import build as obuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = {
    "scale_dropped": ("sbuf[a] = P->scale * dot_qk(P, bh, i, jbuf[a]);", "sbuf[a] = dot_qk(P, bh, i, jbuf[a]);"),
    "lse_sign": ("*lse = m + log(z);", "*lse = m - log(z);"),
    "max_added": ("z += exp(sbuf[a] - m);", "z += exp(sbuf[a] + m);"),
    "strided_a1_bound": ("int64_t t = imax(0, i - l); /* A1", "int64_t t = imax(0, i - l + 1); /* A1"),
    "fixed_a2_first_column": ("cnt = put_range(out, cnt, L * l + w, imin(L * l + w + c - 1, i));",
                              "cnt = put_range(out, cnt, L * l + w - 1, imin(L * l + w + c - 1, i));"),
    "fixed_shared_window": ("if (pattern != O_FIXED_PER_HEAD) return l - c;", "if (pattern != O_FIXED_PER_HEAD) return l - c - 1;"),
    "fixed_own_block_summary_dropped": ("for (int64_t L = 0; L <= blk; ++L)", "for (int64_t L = 0; L < blk; ++L)"),
    "qk_row_swapped": ("int64_t qi = row_base(P, bh, i), kj = row_base(P, bh, j);",
                       "int64_t qi = row_base(P, bh, j), kj = row_base(P, bh, i);"),
    "dk_scale_dropped": ("dk[t] += P->scale * ds * load_elem(P->q", "dk[t] += ds * load_elem(P->q"),
    "delta_dropped": ("double ds = p * (dot_dov(P, bh, i, j) - delta);", "double ds = p * dot_dov(P, bh, i, j);"),
    "dv_wrong_operand": ("dv[t] += p * load_elem(P->dout, P->dtype, qi + t);",
                         "dv[t] += p * load_elem(P->q, P->dtype, qi + t);"),
    "col_set_double_count": ("for (int64_t i = j + 2 * l; i < n; i += l) {", "for (int64_t i = j + l; i < n; i += l) {"),
    "interleave_swapped": ("return (h % 2 == 0) ? O_PART_A1 : O_PART_A2;", "return (h % 2 == 0) ? O_PART_A2 : O_PART_A1;"),
    "empty_row_lse": ("*lse = -INFINITY;", "*lse = 0.0;"),
    "tile_kind_threshold": ("kind[e] = (uint8_t)(cnt[kb] == B * B ? 0 : 1);", "kind[e] = (uint8_t)(cnt[kb] >= B ? 0 : 1);"),
    "per_head_subblock_order": ("return l - (h % (l / c) + 1) * c;", "return (h % (l / c)) * c;"),
    "per_head_window_upper_dropped": ("int summary = (j % l) >= w && (j % l) < w + c;", "int summary = (j % l) >= w;"),
    "per_head_layout_shift": ("s = g == 0 ? 0 : g - 1;", "s = g;"),
    "transpose_row_index": ("row_idx[pos] = (int32_t)qb;", "row_idx[pos] = (int32_t)col_idx[e];"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(obuild.SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    msrc = tmp_path / "mutant.c"
    msrc.write_text(src.replace(old, new))
    mlib = obuild.build(src=str(msrc), lib=str(tmp_path / "libmutant.so"))
    env = dict(os.environ, SPARSE_ATTN_ORACLE_LIB=mlib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "tests/test_oracle_pins.py", "tests/test_oracle_layout.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"
