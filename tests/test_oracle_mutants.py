"""Plant plausible mistakes in copies of the oracle (CPU only) and check that the
pin battery catches every one of them: evidence that the pins constrain each
part of the oracle (gate matrices, orientation, expectation, adjoint sweep,
gradient accumulation, parameter shift, shot sampling, controlled rotations,
embeddings, Pauli-channel trajectories)."""

import os
import shutil

import pytest

import oracle
import oracle_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

# (name, original text, replacement)
MUTANTS = [
    ("ry_sign", "m[1] = -s; m[2] = s;", "m[1] = s; m[2] = -s;"),
    ("full_angle", "double c = cos(0.5 * theta), s = sin(0.5 * theta);",
     "double c = cos(theta), s = sin(theta);"),
    ("rx_sign", "m[1] = -I * s; m[2] = -I * s;", "m[1] = I * s; m[2] = I * s;"),
    ("rz_phases_swapped", "m[0] = c - I * s; m[1] = 0; m[2] = 0; m[3] = c + I * s;",
     "m[0] = c + I * s; m[1] = 0; m[2] = 0; m[3] = c - I * s;"),
    ("h_sign", "m[2] = r; m[3] = -r;", "m[2] = -r; m[3] = r;"),
    ("cnot_orientation", "const int64_t cb = (int64_t)1 << c, tb = (int64_t)1 << t;",
     "const int64_t cb = (int64_t)1 << t, tb = (int64_t)1 << c;"),
    ("cz_any_bit", "if ((j & ab) == ab) psi[j] = -psi[j];", "if (j & ab) psi[j] = -psi[j];"),
    ("transposed_operand", "psi[j] = m[0] * a + m[1] * b;\n        psi[j | bit] = m[2] * a + m[3] * b;",
     "psi[j] = m[0] * a + m[2] * b;\n        psi[j | bit] = m[1] * a + m[3] * b;"),
    ("expect_sign", "return (j & c->bit) ? -p : p;", "return (j & c->bit) ? p : -p;"),
    ("expect_wrong_qubit", "term_ctx c = { psi, NULL, (int64_t)1 << q, 0, 0, NULL };",
     "term_ctx c = { psi, NULL, (int64_t)1 << (q ^ 1), 0, 0, NULL };"),
    ("no_dagger", "if (dagger) { adjoint2(m, a);", "if (0) { adjoint2(m, a);"),
    ("dagger_without_transpose", "a[0] = conj(m[0]); a[1] = conj(m[2]);\n    a[2] = conj(m[1]);",
     "a[0] = conj(m[0]); a[1] = conj(m[1]);\n    a[2] = conj(m[2]);"),
    ("re_instead_of_im", "return cimag(conj(c->lam[j]) * pj);", "return creal(conj(c->lam[j]) * pj);"),
    ("y_generator_sign", "case G_RY: pj = (j & b) ? I * c->psi[j ^ b] : -I * c->psi[j ^ b]; break;",
     "case G_RY: pj = (j & b) ? -I * c->psi[j ^ b] : I * c->psi[j ^ b]; break;"),
    ("x_generator_as_z", "case G_RX: pj = c->psi[j ^ b]; break;", "case G_RX: pj = c->psi[j]; break;"),
    ("seed_sign", "d += ((j >> q) & 1) ? -g_b[q] : g_b[q];", "d += ((j >> q) & 1) ? g_b[q] : -g_b[q];"),
    ("shared_param_overwrite", "if (gk->src == SRC_WEIGHT) { if (grad_w) grad_w[gk->index] += v; }",
     "if (gk->src == SRC_WEIGHT) { if (grad_w) grad_w[gk->index] = v; }"),
    # psi one gate behind lambda in the inner product (un-applying both first
    # would be equivalent: a rotation commutes with its own generator)
    ("psi_lambda_misaligned",
     "double v = im_inner(lam, psi, dim, gk);",
     "apply_gate(psi, dim, gk, th, 0, 1);\n"
     "                double v = im_inner(lam, psi, dim, gk);\n"
     "                apply_gate(psi, dim, gk, th, 0, 0);"),
    ("shift_without_half", "d = 0.5 * (f[0] - f[1]);", "d = (f[0] - f[1]);"),
    ("lambda_not_unapplied", "            apply_gate(lam, dim, gk, th, which, 1);\n", "\n"),
    ("sample_ge_instead_of_gt", "if (cdf[mid] > r) hi = mid;", "if (cdf[mid] >= r) hi = mid;"),
    ("sample_off_by_one", "out[(size_t)b * (size_t)shots + (size_t)s] = lo;",
     "out[(size_t)b * (size_t)shots + (size_t)s] = lo > 0 ? lo - 1 : 0;"),
    ("sample_amplitude_not_squared", "acc += p[2 * j] * p[2 * j] + p[2 * j + 1] * p[2 * j + 1];",
     "acc += fabs(p[2 * j]) + fabs(p[2 * j + 1]);"),
    ("sample_unscaled_uniform", "const double r = u[(size_t)b * (size_t)shots + (size_t)s] * acc;",
     "const double r = u[(size_t)b * (size_t)shots + (size_t)s];"),
    ("crot_ignores_control", "if ((j & bit) || (j & cmask) != cmask) continue;", "if (j & bit) continue;"),
    ("crot_grad_all_amplitudes", "    if (c->cbit && !(j & c->cbit)) return 0.0;\n", ""),
    ("crot_control_target_swapped", "apply_matrix(psi, dim, (int64_t)1 << g->q0, g->q1, m);",
     "apply_matrix(psi, dim, (int64_t)1 << g->q1, g->q0, m);"),
    ("crot_two_term_shift", "const int ns = is_crot(g[k].kind) ? 4 : 2;", "const int ns = 2;"),
    ("four_term_second_sign", "- (r2 - 1) / (4 * r2) * (f[2] - f[3]);", "+ (r2 - 1) / (4 * r2) * (f[2] - f[3]);"),
    ("pauli_y_sign", "else if (which == 2) { psi[j] = -I * b; psi[j | bit] = I * a; }",
     "else if (which == 2) { psi[j] = I * b; psi[j | bit] = -I * a; }"),
    ("pauli_x_as_z", "if (u < c1) return 1;", "if (u < c1) return 3;"),
    ("pauli_edge_in_lower_bin", "if (u < c1) return 1;", "if (u <= c1) return 1;"),
    ("pauli_z_on_bit0", "else psi[j | bit] = -b;", "else psi[j] = -a;"),
    ("pauli_cumulative_missing", "const double c1 = p[0], c2 = c1 + p[1], c3 = c2 + p[2];",
     "const double c1 = p[0], c2 = p[1], c3 = p[2];"),
    ("basis_threshold_strict", "if (x_b[first + q] >= 0.5) idx", "if (x_b[first + q] > 0.5) idx"),
    ("amplitude_unnormalised", "for (int64_t j = 0; j < dim; j++) psi[j] = x_b[first + j] / r;",
     "for (int64_t j = 0; j < dim; j++) psi[j] = x_b[first + j];"),
    ("amplitude_grad_no_projection", "2.0 / r * (creal(lam[j]) - creal(psi[j]) * L);", "2.0 / r * creal(lam[j]);"),
    ("amplitude_grad_half", "2.0 / r * (creal(lam[j])", "1.0 / r * (creal(lam[j])"),
    # the chunked pairwise sum of states of 2^15 amplitudes or more: the tree
    # that combines the chunks stops one level early (half the amplitudes)
    ("pairwise_last_level_dropped", "for (int w = 1; w < nch; w <<= 1)", "for (int w = 1; w < nch / 2; w <<= 1)"),
    # the chunks are laid out with a stride one chunk too short, so the last
    # chunk's amplitudes are never summed and the first are summed twice
    ("pairwise_chunks_misplaced", "part[i] = psum_real(c, f, (int64_t)i * len, (int64_t)(i + 1) * len);",
     "part[i] = psum_real(c, f, (int64_t)i * (len - 1), (int64_t)i * (len - 1) + len);"),
]


@pytest.fixture(scope="module")
def mutant_dir(tmp_path_factory):
    return tmp_path_factory.mktemp("oracle_mutants")


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(mutant_dir, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    path = mutant_dir / f"{name}.c"
    path.write_text(src.replace(old, new))
    lib = oracle.compile_source(str(path), str(mutant_dir / f"lib{name}.so"))
    orc = oracle.Oracle(lib)
    caught = None
    for pin in oracle_pins.ALL_PINS:  # the first pin that fails is enough
        try:
            pin(orc)
        except AssertionError:
            caught = pin.__name__
            break
    assert caught, f"mutant {name} passed every pin"
