"""Planted mistakes in the oracle must be caught by its pins.

Each case rewrites one snippet of one oracle function (a dropped term, a
wrong sign or exponent, a transposed operand, a swapped ratio), installs the
broken function in place of the real one for the duration of the test, and
checks that at least one of the named pins now fails.  This is the evidence
that the pins constrain every part of the oracle and are not tautologies.
"""
import inspect
import textwrap

import pytest

import oracle.shampoo_oracle as O
from tests import oracle_pins as P

MUTATIONS = [
    # (function, original snippet, planted mistake, pins that must notice)
    ("inv_root", "w ** (-1.0 / p)", "w ** (1.0 / p)", [P.pin_root_diagonal]),
    ("inv_root", "w = w + eps_eff", "w = w + 0.0 * eps_eff", [P.pin_root_diagonal]),
    ("inv_root", "(Q * w ** (-1.0 / p)) @ Q.T", "(Q * w ** (-1.0 / p)) @ Q", [P.pin_root_mpmath_4x4]),
    ("sym_eig", "As = 0.5 * (A + A.T)", "As = np.triu(A) + np.triu(A, 1).T",
     [P.pin_root_asymmetric_input, P.pin_cond_damped]),
    ("damping", "return float(eps) * float(lam_max), float(lam_max)",
     "return float(eps), float(lam_max)", [P.pin_root_scaled_identity]),
    ("stats_update", "c * (G @ G.T)", "c * (G.T @ G) if G.shape[0] == G.shape[1] else c * (G @ G.T)",
     [P.pin_stats_integer_bruteforce, P.pin_lemma1]),
    ("stats_update", "c = 1.0 if beta2 == 1.0 else 1.0 - beta2", "c = 1.0", [P.pin_stats_ema]),
    ("stats_update", "beta2 * _f64(R)", "_f64(R)", [P.pin_stats_ema]),
    ("max_sv", "lam_old, lam = lam, float(vh @ v)", "lam_old, lam = lam, float(v @ v)", [P.pin_maxsv]),
    ("coupled_newton", "M1 = (1.0 - alpha) * I + alpha * M", "M1 = (1.0 + alpha) * I - alpha * M",
     [P.pin_newton_vs_eigh]),
    ("coupled_newton", "X = z ** (1.0 / p) * I", "X = z ** (-1.0 / p) * I", [P.pin_newton_vs_eigh]),
    ("coupled_newton", "M = np.linalg.matrix_power(M1, p) @ M", "M = np.linalg.matrix_power(M1, p - 1) @ M",
     [P.pin_newton_vs_eigh]),
    ("coupled_newton", "z = (1.0 + p) / (2.0 * np.linalg.norm(Ad, 'fro'))",
     "z = (1.0 + p) / (2.0 * np.linalg.norm(As, 'fro'))", [P.pin_newton_scalar_iters]),
    ("coupled_newton", "np.linalg.matrix_power(z * Ad, 4), 'fro') ** 0.25", "np.linalg.matrix_power(z * Ad, 2), 'fro') ** 0.5",
     [P.pin_newton_power4_scaling]),
    ("coupled_newton", "z *= max(1.0, (1.0 + p) / (2.0 * rho))", "z *= max(1.0, (1.0 + p) / rho)",
     [P.pin_newton_power4_scaling]),
    ("coupled_newton_warm", "M = np.linalg.matrix_power(X, p) @ Ad", "M = np.linalg.matrix_power(X, p - 1) @ Ad",
     [P.pin_newton_warm]),
    ("coupled_newton_warm", "X = X @ M1", "X = M1 @ X", [P.pin_newton_warm]),
    ("tensor_stats", "Gi = np.moveaxis(G, i, 0).reshape(G.shape[i], -1)",
     "Gi = G.reshape(G.shape[i], -1)", [P.pin_tensor_stats_bruteforce]),
    ("tensor_stats", "S = beta2 * _f64(stats[i]) + S", "S = _f64(stats[i]) + S", [P.pin_tensor_stats_bruteforce]),
    ("tensor_precondition", "np.tensordot(_f64(H), P, axes=(1, i))", "np.tensordot(_f64(H), P, axes=(0, i))",
     [P.pin_tensor_precondition_kronecker]),
    ("tensor_precondition", "P = np.moveaxis(np.tensordot(_f64(H), P, axes=(1, i)), 0, i)",
     "P = np.tensordot(_f64(H), P, axes=(1, i))",
     [P.pin_tensor_precondition_kronecker]),
    ("coupled_newton_warm", "if r < STAG_GATE and r_new >= r and r_new > tol:",
     "if False and r < STAG_GATE and r_new >= r and r_new > tol:", [P.pin_newton_warm]),
    ("coupled_newton_warm", "if not (c <= comm_tol * scale) or grew >= 2:",
     "if not (c <= 1e6 * comm_tol * scale) or grew >= 2:", [P.pin_newton_warm]),
    ("coupled_newton_warm", "    if aborted:\n        res = coupled_newton(", "    if False:\n        res = coupled_newton(",
     [P.pin_newton_warm]),
    ("precondition", "P = _f64(Lr) @ P", "P = _f64(Lr).T @ P", [P.pin_precondition_kronecker]),
    ("precondition", "P = P @ _f64(Rr)", "P = P @ _f64(Rr).T",
     [P.pin_precondition_kronecker]),
    ("adagrad_direction", "G[nz] / np.sqrt(D[nz])", "G[nz] / D[nz]", [P.pin_graft_norm_identity]),
    ("graft_update", "D = _f64(D) + _f64(G) ** 2", "D = _f64(D) + _f64(G)", [P.pin_graft_norm_identity]),
    ("graft_update", "eta = 0.0 if nps == 0.0 else eta0 * nm / nps", "eta = 0.0 if nm == 0.0 else eta0 * nps / nm",
     [P.pin_graft_norm_identity, P.pin_graft_identity_roots]),
    ("graft_update", "beta1 * _f64(Ps) + (1.0 - beta1) * Pf", "beta1 * _f64(Ps) + Pf", [P.pin_graft_momentum_1x1]),
    ("graft_update", "W_new = W - eta * Mg_new", "W_new = W - eta * G", [P.pin_graft_adagrad_fallback]),
    ("lamb_graft_update", "nw = float(np.linalg.norm(W))", "nw = float(np.linalg.norm(Gf))",
     [P.pin_lamb_step_norm]),
    ("lamb_graft_update", "eta = 0.0 if nd == 0.0 else eta0 * nw / nd", "eta = 0.0 if nd == 0.0 else eta0 * nw",
     [P.pin_lamb_step_norm, P.pin_lamb_worked]),
    ("lamb_graft_update", "beta1 * _f64(Ps) + (1.0 - beta1) * Pf", "beta1 * _f64(Ps) + Pf", [P.pin_lamb_worked]),
    ("lamb_graft_update", "beta1 * _f64(Mg) + (1.0 - beta1) * Gf", "(1.0 - beta1) * Gf", [P.pin_lamb_worked]),
    ("lamb_graft_update", "        direction = Mg_new", "        direction = Gf * 0 + np.sign(Gf)",
     [P.pin_lamb_step_norm]),
    ("embedding_grad", "G[i[e]] += w[e] * dy[f[e]]", "G[i[e]] = w[e] * dy[f[e]]",
     [P.pin_embedding_worked_example, P.pin_embedding_lookup_matrix]),
    ("embedding_grad", "G[i[e]] += w[e] * dy[f[e]]", "G[i[e]] += dy[f[e]]", [P.pin_embedding_worked_example]),
    ("embedding_grad", "G[i[e]] += w[e] * dy[f[e]]", "G[f[e]] += w[e] * dy[i[e] % dy.shape[0]]",
     [P.pin_embedding_worked_example]),
    ("_valid_entries", "(idx >= 0) & (idx < vocab)", "(idx >= -1) & (idx < vocab)",
     [P.pin_embedding_worked_example]),
    ("embedding_rows", "acc[r] += w[e] * dy[f[e]]", "acc[r] = w[e] * dy[f[e]]",
     [P.pin_embedding_lookup_matrix, P.pin_embedding_worked_example]),
    ("embedding_rows", "rows = np.array(sorted(acc), dtype=np.int64)", "rows = np.array(list(acc), dtype=np.int64)",
     [P.pin_embedding_lookup_matrix, P.pin_embedding_worked_example]),
    ("cond_damped", "w = w + eps_eff", "w = w + 0.0 * eps_eff", [P.pin_cond_damped]),
    ("cond_damped", "eps_eff, _ = damping(As, eps, eps_relative, lam_max)", "eps_eff, _ = damping(As, eps, False, lam_max)",
     [P.pin_cond_damped]),
    ("cond_damped", "float(w.max() / w.min())", "float(w.max() / abs(w).max())", [P.pin_cond_damped]),
    ("cond_damped", "As, w, _ = sym_eig(A) if eig is None else eig", "As, w, _ = sym_eig(np.triu(A)) if eig is None else eig",
     [P.pin_cond_damped]),
    ("cond_damped", "if w.min() > 0 else np.inf", "if w.min() != 0 else np.inf", [P.pin_cond_damped]),
    ("shampoo_step", "s['Lr'], st, _ = inv_root(L, p, eps, eps_relative)",
     "s['Lr'], st, _ = inv_root(state['L'] + 0.0 * L, p, eps, eps_relative)",
     [P.pin_shampoo_step_kronecker, P.pin_shampoo_step_variants]),
    ("shampoo_step", "s['Rr'], st, _ = inv_root(R, p, eps, eps_relative)",
     "s['Rr'], st, _ = inv_root(R, p, 0.0, eps_relative)", [P.pin_shampoo_step_kronecker]),
    ("shampoo_step", "P = precondition(G, s.get('Lr') if left else None,\n                     s.get('Rr') if right else None)",
     "P = precondition(G, s.get('Rr') if right else None,\n                     s.get('Lr') if left else None)",
     [P.pin_shampoo_step_kronecker]),
    ("shampoo_step", "    if refresh_roots:", "    if True:", [P.pin_shampoo_step_kronecker]),
    ("shampoo_step", "out = graft_update(s['W'], s['D'], G, P, eta0, beta1,", "out = graft_update(s['W'], s['D'], G, P, eta0, 0.0,",
     [P.pin_shampoo_step_variants]),
    ("shampoo_step", "s.update(W=out['W'], D=out['D'],", "s.update(W=out['W'], D=s['D'],",
     [P.pin_shampoo_step_kronecker]),
    ("bf16_bits_to_f64", "<< 16", "<< 15", [P.pin_bf16_decode]),
    ("bf16_bits_to_f64", "return bits.view(np.float32).astype(np.float64)",
     "return bits.astype(np.float32).astype(np.float64)", [P.pin_bf16_decode]),
    ("bf16_bits_to_f64", "return bits.view(np.float32).astype(np.float64)",
     "return bits.view(np.float32).astype(np.float16).astype(np.float64)", [P.pin_bf16_decode]),
]


def _mutant(fname, old, new):
    src = textwrap.dedent(inspect.getsource(getattr(O, fname)))
    assert old in src, f"snippet not found in {fname}: {old}"
    ns = {}
    exec(compile(src.replace(old, new), f"<mutant {fname}>", "exec"), O.__dict__, ns)
    return ns[fname]


@pytest.mark.parametrize("fname,old,new,pins", MUTATIONS,
                         ids=[f"{m[0]}:{i}" for i, m in enumerate(MUTATIONS)])
def test_planted_mistake_is_caught(monkeypatch, fname, old, new, pins):
    monkeypatch.setattr(O, fname, _mutant(fname, old, new))
    caught = []
    for pin in pins:
        try:
            pin(O)
        except (AssertionError, ValueError, FloatingPointError, ZeroDivisionError, TypeError):
            caught.append(pin.__name__)
    assert caught, f"mutation of {fname} ({new!r}) slipped past {[p.__name__ for p in pins]}"


def test_real_oracle_passes_all_pins_used_here():
    for _, _, _, pins in MUTATIONS:
        for pin in pins:
            pin(O)
