"""First-order rounding-error model of the mixed-precision exit-head step.

Test infrastructure: the GPU parity tests use it to bound every output
element against the fp64 oracle.  It does not run the HIP path and shares
no code with it; it takes the oracle's fp64 intermediates and propagates
the variance that each rounding of the mixed-precision convention adds
(bf16 storage of every tensor a kernel hands to the next, fp32 arithmetic
and accumulation, fp32 weight gradients):

  * one rounding of a value q to nearest even adds an error e q with e
    uniform in [-u, u], variance (u^2 / 3) q^2; u = 2^-8 for bf16 (8
    significant bits).  fp32 storage and fp32 transcendental functions are
    modelled with u = 2^-21 (a few ulp, and the error of the
    exponential's fp32 argument);
  * an error in an operand of a product C = A B^T propagates as
    var(C) = var(A) (B^2)^T + A^2 var(B)^T, with errors of different
    elements taken as independent (weights are random, so the cross terms
    average out); an accumulation over K terms in fp32 adds
    (u32^2 / 3) (K / 2) (A^2 (B^2)^T);
  * elementwise maps propagate through their first derivatives;
  * normalisation propagates r^2 var(input) (the projection it removes only
    lowers the error);
  * one exception to independence: the target entries s_n (p_y - 1) of
    rows with equal s_n are nearly equal numbers, so their roundings err
    alike.  Sums that carry no other factor of random sign (the bias
    gradient, sum_n dZ[n, j]) get the fully correlated term
    (u^2 / 3) (sum_n W[y_n, j] G[n, y_n])^2 per group of equal s_n.

The rounding points follow the precision convention of the boundary
(norms, softmax and losses in fp32; GEMMs on bf16 operands with fp32
accumulation; the logits stored once in bf16 as exp(S - m) and turned into
the bf16 logit-gradient seed G, or, in the unshifted form, stored as
exp(S) with the per-token factor s_n exp(-LSE_n) rounded into the bf16
token-contiguous x_hat and the target entries shifted by exp(LSE_n) in
bf16; weight gradients in fp32).  Both forms round each term P x_hat of a
weight gradient three times (P, then G or x_hat's scaled copy, and x_hat),
so one variance covers both; the unshifted form's dZ = coef (P' W) rounds
less and stays inside it.  The result is a
standard deviation sigma per output element; the tests accept
|gpu - oracle| <= K_SIGMA sigma + floor.  A single dominant term of a sum
is covered as well: its error is at most a few u times the term, while
K_SIGMA sigma is at least K_SIGMA u / sqrt(3) times it.
"""

from __future__ import annotations

from typing import Dict, Optional

import numpy as np

import oracle as O

U_BF16 = 2.0 ** -8
U_F32 = 2.0 ** -21
U_ACC = 2.0 ** -24
K_SIGMA = 8.0


def rnd(q, u):
    """Variance of one rounding of q."""
    return (u * u / 3.0) * q * q


def acc(a2, b2t, k):
    """Variance of a fp32 accumulation of depth k of products A B^T, given
    A^2 and (B^2)^T."""
    return acc_coef(k) * mm(a2, b2t)


def acc_coef(k):
    return (U_ACC * U_ACC / 3.0) * (k / 2.0)


def mm(a, b):
    """Product of two variance-sized arrays.  A variance needs a few
    significant digits, so the full-size products run in fp32; small ones
    run in fp64, whose range also holds the squared rounding errors of
    probabilities far below one (an fp32 variance of an element near 1e-22
    underflows to zero)."""
    a = np.asarray(a)
    b = np.asarray(b)
    if a.size * (b.shape[-1] if b.ndim > 1 else 1) <= 1 << 28:
        return np.asarray(a, dtype=np.float64) @ np.asarray(b, dtype=np.float64)
    return (np.asarray(a, dtype=np.float32) @ np.asarray(b, dtype=np.float32)).astype(np.float64)


def dsilu2(t):
    """Second derivative of silu(t) = t sigmoid(t)."""
    s = O.sigmoid(t)
    return s * (1.0 - s) * (2.0 + t * (1.0 - 2.0 * s))


def step_sigma(e: "O.Exit", x: np.ndarray, y: np.ndarray, exit_weight: float, dtype: str,
               v_rows: Optional[np.ndarray] = None, i_rows: Optional[np.ndarray] = None,
               token_weights: Optional[np.ndarray] = None, dynamic_weights: bool = False,
               chunk: int = O.CHUNK_ROWS) -> Dict[str, np.ndarray]:
    """Standard deviation of the rounding error of every output of one exit.

    Returns sigma for "row_loss" [N] and, by the same names as the oracle's
    gradients, for "w_out" (rows v_rows, or all), "gamma", "beta",
    "gamma_mlp", "w_gate" / "w_up" (rows i_rows, or all) and "w_down"
    (columns i_rows, or all).
    """
    u = U_BF16 if dtype == "bf16" else U_F32
    n_all = x.shape[0]
    V, h = e.w_out.shape
    vr = np.arange(V) if v_rows is None else np.asarray(v_rows)
    mlp = e.kind == O.EXIT_MLP
    if mlp:
        I = e.w_gate.shape[0]
        ir = np.arange(I) if i_rows is None else np.asarray(i_rows)
    W = e.w_out
    W2 = W * W
    var: Dict[str, np.ndarray] = {}
    row = np.empty(n_all)
    coherent: Dict[float, np.ndarray] = {}     # bias gradient: per value of s_n

    def add(k, v):
        var[k] = v if k not in var else var[k] + v

    for r0 in range(0, n_all, chunk):
        r1 = min(n_all, r0 + chunk)
        xs = x[r0:r1]
        n = r1 - r0
        f = O.exit_forward(e, xs)
        s = f["s"]
        lse = O.log_sum_exp(s)
        p = np.exp(s - lse[:, None])
        conf = O.confidence(s)
        m = O.row_weights(conf, token_weights, r0, r1, dynamic_weights)
        sn = exit_weight * m / n_all
        onehot = np.zeros_like(p)
        onehot[np.arange(n), y[r0:r1]] = 1.0
        G = sn[:, None] * (p - onehot)

        # ------------------------------------------------------- forward
        if mlp:
            u_hat, uu, hg, hu, a = f["u_hat"], f["u"], f["hg"], f["hu"], f["a"]
            v_u = rnd(uu, u)
            v_uhat = rnd(u_hat, u)
            v_uacc = v_u + acc_coef(h) * uu * uu
            v_hg = mm(v_uacc, (e.w_gate ** 2).T) + rnd(hg, u)
            v_hu_acc = mm(v_uacc, (e.w_up ** 2).T)
            v_hu = v_hu_acc + rnd(hu, u)
            sg = O.silu(hg)
            dsg = O.silu_grad(hg)
            v_a = (dsg * hu) ** 2 * v_hg + sg ** 2 * v_hu_acc + rnd(a, u)
            wd2 = e.w_down ** 2
            v_y = mm(v_a + acc_coef(I) * a * a, wd2.T)
            r = f["r"]
            zh = f["z_hat"]
            v_zh = (r * r)[:, None] * v_y + rnd(zh, u)                 # stored Z_hat (weight gradients)
            v_z = (r * r)[:, None] * v_y * (e.gamma ** 2)[None, :] + rnd(f["z"], u)
        elif e.kind == O.EXIT_NORM:
            zh = f["z_hat"]
            v_zh = rnd(zh, u)
            v_z = rnd(f["z"], u)
        else:
            zh = None
            v_z = np.zeros_like(xs)           # Z = X, exact
            v_zh = v_z
        z = f["z"]
        # logits: S = Z W^T (fp32 accumulation); a = E_p[W] per row
        v_zacc = v_z + acc_coef(h) * z * z
        a_row = mm(p, W)
        # var(dS_v - dLSE) = sum_j var(Z)_j (W_vj - a_j)^2
        v_sml = mm(v_zacc, W2.T) - 2.0 * mm(v_zacc * a_row, W.T) + np.sum(v_zacc * a_row * a_row, axis=1)[:, None]
        v_sml = np.maximum(v_sml, 0.0) + (16 * U_ACC) ** 2          # fp32 LSE from the partials
        # per-row NLL: sum_v p_v dS_v - dS_y
        d = a_row - W[y[r0:r1]]
        row[r0:r1] = np.sqrt(np.sum(v_z * d * d, axis=1) + (16 * U_ACC) ** 2 * (1.0 + lse ** 2)
                             + (U_ACC * np.abs(s[np.arange(n), y[r0:r1]])) ** 2)
        # seed G = s_n (p - onehot): roundings of P = exp(S - m) and of G, the
        # logit error, and (dynamic weights) the error of the confidence
        v_g = (sn[:, None] * p) ** 2 * (u * u / 3.0 + v_sml) + rnd(G, u)
        if dynamic_weights:
            amax = np.argmax(s, axis=1)
            dm = W[amax] - a_row
            v_c = np.sum(v_z * dm * dm, axis=1) + (16 * U_ACC) ** 2
            v_g = v_g + G * G * v_c[:, None]
        # ------------------------------------------------------ backward
        G2 = G * G
        if e.kind == O.EXIT_EMBEDDING:
            add("w_out", mm((v_g[:, vr] + acc_coef(n) * G2[:, vr]).T, z * z))
            continue
        zh2 = zh * zh
        gam2 = e.gamma ** 2
        add("w_out", gam2[None, :] * (mm((v_g[:, vr] + acc_coef(n) * G2[:, vr]).T, zh2) + mm(G2[:, vr].T, v_zh)))
        if e.beta is not None:
            # dW += (sum_n G_nv) beta_j
            add("w_out", np.sum(v_g[:, vr], axis=0)[:, None] * (e.beta ** 2)[None, :])
        dz = mm(G, W)
        v_dz = mm(v_g + acc_coef(V) * G2, W2)       # var(dZ): dZ = G W in fp32
        add("gamma", np.sum(zh2 * v_dz + v_zh * dz * dz, axis=0))
        if e.beta is not None:
            # bias gradient: sum_v W_vj (sum_n G_nv)
            add("beta", np.sum(v_dz, axis=0))
            yy = y[r0:r1]
            gy = G[np.arange(n), yy]
            vals, inv = np.unique(sn, return_inverse=True)
            for k_, sv in enumerate(vals):
                sel = inv == k_
                t = gy[sel] @ W[yy[sel]]
                coherent[float(sv)] = t if float(sv) not in coherent else coherent[float(sv)] + t
        if not mlp:
            continue
        # the exit-norm backward of dZ and its bf16 dY
        gam = e.gamma
        dzh = dz * gam[None, :]
        dy = O.rmsnorm_backward(dzh, zh, r)
        proj = np.mean(dzh * zh, axis=1)
        v_dy = (r * r)[:, None] * (gam2[None, :] * v_dz + (proj * proj)[:, None] * (r * r)[:, None] * v_y) \
            + rnd(dy, u)
        # dA = dY W_d; the SwiGLU backward; the down-projection gradient
        da = mm(dy, e.w_down)
        v_da = mm(v_dy + acc_coef(h) * dy * dy, wd2)
        d_hg = da * hu * dsg
        d_hu = da * sg
        v_dhg = (hu * dsg) ** 2 * v_da + (da * dsg) ** 2 * v_hu + (da * hu * dsilu2(hg)) ** 2 * v_hg \
            + rnd(d_hg, u)
        v_dhu = sg ** 2 * v_da + (da * dsg) ** 2 * v_hg + rnd(d_hu, u)
        add("w_down", mm((v_dy + acc_coef(n) * dy * dy).T, a[:, ir] ** 2) + mm((dy * dy).T, v_a[:, ir]))
        gm2 = e.gamma_mlp ** 2
        uh2 = u_hat * u_hat
        add("w_gate", gm2[None, :] * (mm((v_dhg[:, ir] + acc_coef(n) * d_hg[:, ir] ** 2).T, uh2)
                                      + mm((d_hg[:, ir] ** 2).T, v_uhat)))
        add("w_up", gm2[None, :] * (mm((v_dhu[:, ir] + acc_coef(n) * d_hu[:, ir] ** 2).T, uh2)
                                    + mm((d_hu[:, ir] ** 2).T, v_uhat)))
        wg2, wu2 = e.w_gate ** 2, e.w_up ** 2
        du = mm(d_hg, e.w_gate) + mm(d_hu, e.w_up)
        c_i = acc_coef(I)
        add("gamma_mlp", np.sum(uh2 * (mm(v_dhg + c_i * d_hg ** 2, wg2) + mm(v_dhu + c_i * d_hu ** 2, wu2))
                                + v_uhat * du * du, axis=0))
    if coherent:
        var["beta"] = var["beta"] + (u * u / 3.0) * sum(t * t for t in coherent.values())
    out = {k: np.sqrt(np.maximum(v, 0.0)) for k, v in var.items()}
    out["row_loss"] = row
    return out


def check_elementwise(label: str, got: np.ndarray, ref: np.ndarray, sigma: np.ndarray,
                      floor: float = 0.0, k: float = K_SIGMA) -> float:
    """Assert |got - ref| <= k sigma + floor elementwise; return the largest
    ratio |got - ref| / (k sigma + floor) (at most 1 when it passes)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    bound = k * sigma + floor
    err = np.abs(got - ref)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(bound > 0, err / bound, np.where(err > 0, np.inf, 0.0))
    worst = float(np.max(ratio)) if ratio.size else 0.0
    if not worst <= 1.0:
        idx = np.unravel_index(int(np.argmax(ratio)), ratio.shape)
        raise AssertionError(f"{label}: element {idx} differs by {err[idx]:.3e}, bound {bound[idx]:.3e} "
                             f"(gpu {got[idx]:.6e}, oracle {ref[idx]:.6e}); {int(np.sum(ratio > 1))} elements out")
    return worst
