"""Planted mistakes in the oracle must be caught by its pins (CPU only).

Each case compiles a copy of the oracle source with one plausible mistake (a
dropped term, a wrong sign, a transposed operand, a wrong index or bound) into
a temporary library and runs the pin tests against it in a subprocess; the pins
must fail.  The real oracle is never modified.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "scn_oracle.cpp")

MUTANTS = [
    ("fwd_drop_bias",
     "for (int co = 0; co < Cout; ++co) yo[co] = bias ? bias[co] : 0.0;",
     "for (int co = 0; co < Cout; ++co) yo[co] = 0.0;"),
    ("fwd_inactive_is_zero",
     "q[ci] = r >= 0 ? x[(int64_t)r * Cin + ci] : g_in[ci];\n      for (int ci = 0; ci < Cin; ++ci)\n        for",
     "q[ci] = r >= 0 ? x[(int64_t)r * Cin + ci] : 0.0;\n      for (int ci = 0; ci < Cin; ++ci)\n        for"),
    ("offset_axes_swapped",
     "*kx = c % f;\n    *ky = (c / f) % f;\n    *kz = c / (f * f);",
     "*kz = c % f;\n    *ky = (c / f) % f;\n    *kx = c / (f * f);"),
    ("bwd_dW_drops_ground_term", "gW[w] += g_in[ci] * dgb[co];", "gW[w] += 0.0;"),
    ("bwd_dg_drops_inactive_term", "          gg[ci] += back;", "          gg[ci] += 0.0;"),
    ("pool_keeps_last_max", "if (bk < 0 || v > best)", "if (bk < 0 || v >= best)"),
    ("pool_bwd_drops_ground", "        gg[c] += dy[o * C + c];", "        gg[c] += 0.0;"),
    ("extent_off_by_one", "return m >= f ? (m - f) / s + 1 : 0;", "return m >= f ? (m - f) / s : 0;"),
    ("fwd_W_transposed",
     "yo[co] += q[ci] * W[((int64_t)k * Cin + ci) * Cout + co];",
     "yo[co] += q[ci] * W[((int64_t)k * Cout + co) * Cin + ci];"),
    ("ground_state_sign",
     "gpre[co] += g_in[ci] * W[((int64_t)k * Cin + ci) * Cout + co];",
     "gpre[co] -= g_in[ci] * W[((int64_t)k * Cin + ci) * Cout + co];"),
    ("duplicates_accepted",
     "if (!rb->H_in.emplace(key, static_cast<int32_t>(r)).second) {",
     "if (!rb->H_in.emplace(key, static_cast<int32_t>(r)).second && false) {"),
    ("range_check_off_by_one", "c[1] < 0 || c[1] >= g.mx", "c[1] < 0 || c[1] > g.mx"),
    ("stride_divisibility_dropped",
     "ok = ok && d[a] >= 0 && d[a] % s == 0 && d[a] / s < m[a];",
     "ok = ok && d[a] >= 0 && d[a] / s < m[a];"),
    ("bwd_relu_mask_dropped", "dyb[co] = (relu && !(pre[co] > 0.0)) ? 0.0 : d;", "dyb[co] = d;"),
    ("bwd_dbias_drops_ground", "for (int co = 0; co < Cout; ++co) gB[co] += dgb[co];",
     "for (int co = 0; co < Cout; ++co) gB[co] += 0.0;"),
    ("rules_not_ordered_by_output",
     "rb->lists[k].emplace_back(r, static_cast<int32_t>(o));",
     "rb->lists[k].insert(rb->lists[k].begin(), {r, static_cast<int32_t>(o)});"),
]


# mistakes in the tetrahedral lattice (section 1.2), caught by its own pins
LATTICE_MUTANTS = [
    ("tetra_filter_one_too_big", "if (!simplex || kx + ky + kz < f)",
     "if (!simplex || kx + ky + kz <= f)"),
    ("tetra_output_bound_dropped", "if (simplex) ok = ok && (d[0] + d[1] + d[2]) / s < go.mx;",
     "if (simplex) ok = ok;"),
    ("tetra_output_bound_off_by_one", "if (simplex) ok = ok && (d[0] + d[1] + d[2]) / s < go.mx;",
     "if (simplex) ok = ok && (d[0] + d[1] + d[2]) / s <= go.mx;"),
    ("tetra_range_check_dropped", "(simplex && (int64_t)c[1] + c[2] + c[3] >= g.mx)",
     "(simplex && false)"),
    ("tetra_offsets_reversed", "rb->K = static_cast<int>(rb->offs.size());",
     "std::reverse(rb->offs.begin(), rb->offs.end());\n  rb->K = static_cast<int>(rb->offs.size());"),
]

# mistakes in the 2D lattices (Figure 2 (i), (ii)), caught by their pins
PLANAR_MUTANTS = [
    ("planar_filter_spans_z", "const int fz = planar ? 1 : f;", "const int fz = f;"),
    ("planar_extra_planes_accepted", "if (planar && g.mz != 1) return INVALID;",
     "if (planar && g.mz < 1) return INVALID;"),
    ("triangle_is_square", "const bool simplex = lattice == 1 || lattice == 3;",
     "const bool simplex = lattice == 1;"),
]

# mistakes in the hypercubic lattice of d dimensions (section 1.2), caught by
# its own pins
ND_MUTANTS = [
    ("nd_offset_digits_reversed",
     "for (int a = 0; a < D; ++a) x[a] = s * (int64_t)c[1 + a] + offset_nd(k, a, f);",
     "for (int a = 0; a < D; ++a) x[a] = s * (int64_t)c[1 + a] + offset_nd(k, D - 1 - a, f);"),
    ("nd_key_axes_reversed",
     "for (int a = D - 1; a >= 0; --a) key = key * static_cast<uint64_t>(m[a])",
     "for (int a = 0; a < D; ++a) key = key * static_cast<uint64_t>(m[a])"),
    ("nd_rules_not_ordered_by_output",
     "rb->lists[k].push_back({r, static_cast<int32_t>(o)});",
     "rb->lists[k].insert(rb->lists[k].begin(), {r, static_cast<int32_t>(o)});"),
    ("nd_stride_divisibility_dropped",
     "ok = ok && d >= 0 && d % s == 0 && d / s < rb->m_out[a];",
     "ok = ok && d >= 0 && d / s < rb->m_out[a];"),
    ("nd_last_axis_range_unchecked",
     "ok = ok && x[a] >= 0 && x[a] < rb->m_in[a];",
     "ok = ok && x[a] >= 0 && (a == D - 1 || x[a] < rb->m_in[a]);"),
]

CASES = [m + ("test_oracle_pins.py",) for m in MUTANTS] + \
        [m + ("test_oracle_nd.py",) for m in ND_MUTANTS] + \
        [m + ("test_oracle_lattice.py",) for m in LATTICE_MUTANTS] + \
        [m + ("test_oracle_lattice2d.py",) for m in PLANAR_MUTANTS]


@pytest.mark.parametrize("name,old,new,pins", CASES, ids=[m[0] for m in CASES])
def test_pins_catch_planted_mistake(name, old, new, pins, tmp_path):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique/present"
    mut = tmp_path / "mut.cpp"
    mut.write_text(src.replace(old, new))
    lib = tmp_path / "libmut.so"
    subprocess.run(["g++", "-O1", "-std=c++17", "-shared", "-fPIC", str(mut), "-o", str(lib)],
                   check=True)
    env = dict(os.environ, SCN_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", pins)],
                       env=env, capture_output=True, text=True, cwd=ROOT, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"
