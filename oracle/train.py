"""One FP64 training step of PaiNN on energies and forces (oracle; test
infrastructure only).

The paper trains its lead model (Table "Lead PaiNN model configuration") with
an MAE loss on energies and forces, force weight about 94.8, the AdamW
optimizer at learning rate 6.34e-4, 25 structures per GPU, in FP64 (section
"Flagship Training of Top HPO Models").  It does not write the loss out; the
reading used here (R30) is

  L = (1/B) sum_b |E_b - E*_b| + lambda (1/(3N)) sum_{i,c} |F_ic - F*_ic|

over a batch of B structures with N atoms in total, F = -dE/dx.  Its
gradient with respect to every weight theta is

  dL/dtheta = sum_b c_b dE_b/dtheta - d/dtheta ( sum_i u_i . dE/dx_i )
  c_b = sign(E_b - E*_b) / B,   u_ic = lambda sign(F_ic - F*_ic) / (3N)

(the signs are held fixed: MAE is differentiable wherever no residual is
exactly zero).  The first term is reverse-mode differentiation of the energy
with respect to the weights (`energy_weight_grad`).  The second is the
derivative of that same weight gradient along the position direction u:
dE/dtheta is evaluated at complex positions x + i h u, and its imaginary part
divided by h is d/dh dE/dtheta (x + h u) at h = 0 = d/dtheta (u . dE/dx), to
rounding (the complex-step derivative, Squire & Trapp, SIAM Review 1998).  No
difference is taken, so h = 1e-30 leaves no truncation error; this needs every
step of the energy's weight gradient to be analytic in x, so no absolute
values or branches on complex values appear below (branches test the real
part).  The radius graph is built from the real positions and held fixed.

AdamW (Loshchilov & Hutter, "Decoupled Weight Decay Regularization", ICLR
2019), as `adamw_step`: decay theta <- theta (1 - lr wd), then
m <- b1 m + (1-b1) g, v <- b2 v + (1-b2) g^2, theta <- theta - lr mhat /
(sqrt(vhat) + eps) with mhat = m/(1-b1^t), vhat = v/(1-b2^t); every array
is decayed (R31: the paper gives lr only; b1 = 0.9, b2 = 0.999, eps = 1e-8,
wd = 0.01 are the common defaults of the method).
"""
from __future__ import annotations

import numpy as np

from .forces import structure_forces
from .neighbors import radius_graph

COMPLEX_STEP = 1e-30


def _silu(x):
    return x / (1.0 + np.exp(-x))


def _dsilu(x):
    sg = 1.0 / (1.0 + np.exp(-x))
    return sg * (1.0 + x * (1.0 - sg))


def _basis(d, hp):
    """Radial basis g_k(d) (R6 Gaussian / R24 Bessel), analytic in d."""
    K, rc = hp.K, hp.cutoff
    if hp.rbf_type == 0:
        delta = rc / (K - 1)
        mu = np.arange(K, dtype=np.float64) * delta
        gamma = 1.0 / (2.0 * delta * delta)
        x = d[:, None] - mu
        return np.exp(-gamma * x * x)
    n = np.arange(1, K + 1, dtype=np.float64)
    return np.sin(n * (np.pi / rc) * d[:, None]) / d[:, None]


def _dense(x, w, b):
    return x @ w.T + b


def energy_weight_grad(pos, species, cell, pbc, dataset_id, hp, W, graph=None):
    """Energy E of one structure and dE/dW by a reverse pass in the order of
    the forward, for the arrays E depends on: the embedding, every layer, the
    shared head layers and the structure's own branch (the other branches'
    gradients are zero and left out of the returned dict).  `pos` may be
    complex (the complex step); the graph (recv, send, shift) is that of the
    real positions.  Returns (E, grads)."""
    F = hp.F
    z = np.asarray(species)
    x = np.asarray(pos)
    n = len(z)
    if graph is None:
        graph = radius_graph(np.real(x), cell, pbc, hp.cutoff, getattr(hp, "max_neighbors", 0))
    recv, send, shift = graph
    a = np.asarray(cell, dtype=np.float64).reshape(3, 3)
    sh = shift.astype(np.float64)
    t = (sh[:, 0:1] * a[0][None, :] + sh[:, 1:2] * a[1][None, :]) + sh[:, 2:3] * a[2][None, :]
    r = (x[send] - x[recv]) + t
    d = np.sqrt((r[:, 0] * r[:, 0] + r[:, 1] * r[:, 1]) + r[:, 2] * r[:, 2])
    rhat = r / d[:, None]
    g = _basis(d, hp)                                        # [E, K]
    fc = 0.5 * (np.cos(np.pi * d / hp.cutoff) + 1.0)         # every edge has d < r_c
    dt = np.result_type(x.dtype, np.float64)

    # forward, keeping every intermediate the reverse pass reads
    s = W["emb"][z].astype(dt)
    v = np.zeros((n, 3, F), dtype=dt)
    saved = []
    for l in range(hp.L):
        p = f"l{l}."
        z1 = _dense(s, W[p + "phi_w1"], W[p + "phi_b1"])
        a1 = _silu(z1)
        h = _dense(a1, W[p + "phi_w2"], W[p + "phi_b2"])
        lin = _dense(g, W[p + "filt_w"], W[p + "filt_b"])
        w = fc[:, None] * lin
        hj = h[send]
        s_mid = s.copy()
        v_mid = v.copy()
        np.add.at(s_mid, recv, hj[:, :F] * w[:, :F])
        np.add.at(v_mid, recv, v[send] * (hj[:, None, F:2 * F] * w[:, None, F:2 * F])
                  + rhat[:, :, None] * (hj[:, None, 2 * F:] * w[:, None, 2 * F:]))
        U = v_mid @ W[p + "U"].T
        V = v_mid @ W[p + "V"].T
        n2 = np.sum(V * V, axis=1)
        nz = np.real(n2) > 0
        nrm = np.where(nz, np.sqrt(np.where(nz, n2, 1.0)), 0.0)
        xin = np.concatenate([s_mid, nrm], axis=1)
        za = _dense(xin, W[p + "upd_w1"], W[p + "upd_b1"])
        aa = _silu(za)
        ga = _dense(aa, W[p + "upd_w2"], W[p + "upd_b2"])
        a_vv, a_sv, a_ss = ga[:, :F], ga[:, F:2 * F], ga[:, 2 * F:]
        saved.append(dict(s=s, v=v, z1=z1, a1=a1, h=h, lin=lin, w=w, s_mid=s_mid, v_mid=v_mid, U=U, V=V,
                          nrm=nrm, nz=nz, xin=xin, za=za, aa=aa, a_vv=a_vv, a_sv=a_sv))
        v = v_mid + a_vv[:, None, :] * U
        s = s_mid + a_sv * np.sum(U * V, axis=1) + a_ss
    # heads: shared layers, then the dataset's branch
    names = [(f"shared{m}.w", f"shared{m}.b") for m in range(len(hp.shared_dims))]
    names += [(f"head{dataset_id}.{m}.w", f"head{dataset_id}.{m}.b") for m in range(len(hp.branch_dims))]
    ins, pre = [], []
    y = s
    for m, (wn, bn) in enumerate(names):
        ins.append(y)
        zm = _dense(y, W[wn], W[bn])
        pre.append(zm)
        y = _silu(zm) if m < len(names) - 1 else zm
    E = np.sum(y[:, 0])

    used = ["emb"] + [k for k in W if k.startswith("l") or k.startswith("shared")]
    used += [wn for wn, _ in names] + [bn for _, bn in names]
    G = {k: np.zeros(np.shape(W[k]), dtype=dt) for k in dict.fromkeys(used)}
    # reverse through the heads (dE/de_i = 1)
    gz = np.ones((n, 1), dtype=dt)
    for m in range(len(names) - 1, -1, -1):
        wn, bn = names[m]
        G[wn] += gz.T @ ins[m]
        G[bn] += gz.sum(axis=0)
        gy = gz @ W[wn]
        gz = gy * _dsilu(pre[m - 1]) if m > 0 else gy
    gs = gz
    gv = np.zeros((n, 3, F), dtype=dt)
    for l in range(hp.L - 1, -1, -1):
        p = f"l{l}."
        S = saved[l]
        U, V, a_vv, a_sv = S["U"], S["V"], S["a_vv"], S["a_sv"]
        # update block
        g_a = np.concatenate([np.sum(gv * U, axis=1), gs * np.sum(U * V, axis=1), gs], axis=1)
        G[p + "upd_w2"] += g_a.T @ S["aa"]
        G[p + "upd_b2"] += g_a.sum(axis=0)
        g_za = (g_a @ W[p + "upd_w2"]) * _dsilu(S["za"])
        G[p + "upd_w1"] += g_za.T @ S["xin"]
        G[p + "upd_b1"] += g_za.sum(axis=0)
        g_in = g_za @ W[p + "upd_w1"]
        safe = np.where(S["nz"], S["nrm"], 1.0)
        gU = gv * a_vv[:, None, :] + (gs * a_sv)[:, None, :] * V
        gV = (gs * a_sv)[:, None, :] * U + np.where(S["nz"], g_in[:, F:] / safe, 0.0)[:, None, :] * V
        gs = gs + g_in[:, :F]
        vm = S["v_mid"]
        G[p + "U"] += np.einsum("ncf,nck->fk", gU, vm)
        G[p + "V"] += np.einsum("ncf,nck->fk", gV, vm)
        gv = gv + gU @ W[p + "U"] + gV @ W[p + "V"]
        # message (the residual paths pass gs, gv on)
        h, w, vs = S["h"], S["w"], S["v"]
        gsi, gvi = gs[recv], gv[recv]
        hs, hv, hr = h[send, :F], h[send, F:2 * F], h[send, 2 * F:]
        A_v = np.sum(gvi * vs[send], axis=1)
        A_r = np.sum(gvi * rhat[:, :, None], axis=1)
        g_h = np.zeros((n, 3 * F), dtype=dt)
        np.add.at(g_h, send, np.concatenate([gsi * w[:, :F], A_v * w[:, F:2 * F], A_r * w[:, 2 * F:]], axis=1))
        gv_new = gv.copy()
        np.add.at(gv_new, send, gvi * (hv * w[:, F:2 * F])[:, None, :])
        g_lin = fc[:, None] * np.concatenate([gsi * hs, A_v * hv, A_r * hr], axis=1)
        G[p + "filt_w"] += g_lin.T @ g
        G[p + "filt_b"] += g_lin.sum(axis=0)
        # phi
        G[p + "phi_w2"] += g_h.T @ S["a1"]
        G[p + "phi_b2"] += g_h.sum(axis=0)
        g_z1 = (g_h @ W[p + "phi_w2"]) * _dsilu(S["z1"])
        G[p + "phi_w1"] += g_z1.T @ S["s"]
        G[p + "phi_b1"] += g_z1.sum(axis=0)
        gs = gs + g_z1 @ W[p + "phi_w1"]
        gv = gv_new
    np.add.at(G["emb"], z, gs)
    return E, G


def structure_loss_grad_terms(pos, species, cell, pbc, dataset_id, hp, W, c, u):
    """sum of c dE/dtheta - d/dtheta (u . dE/dx) for one structure (c a
    scalar, u [n, 3]), from one complex evaluation of the weight gradient at
    x + i h u: its real part is dE/dtheta, its imaginary part / h the
    directional derivative."""
    x = np.asarray(pos, dtype=np.float64)
    graph = radius_graph(x, cell, pbc, hp.cutoff, getattr(hp, "max_neighbors", 0))
    h = COMPLEX_STEP
    _, Gc = energy_weight_grad(x + 1j * h * np.asarray(u, dtype=np.float64), species, cell, pbc, dataset_id,
                               hp, W, graph=graph)
    return {k: c * np.real(val) - np.imag(val) / h for k, val in Gc.items()}


def loss_and_grad(batch, hp, W, E_ref, F_ref, force_weight: float):
    """Loss (R30) and its gradient with respect to every weight for a batch.
    Returns dict(loss, loss_E, loss_F, E [B], F [N, 3], grad {name: array})."""
    B, N = batch.n_struct, batch.n_atoms
    E = np.zeros(B)
    Fo = np.zeros((N, 3))
    ds = []
    for b in range(B):
        pos, z, cell, pbc, d = batch.structure(b)
        di = int(d) if hp.n_heads > 1 else 0
        ds.append(di)
        o = structure_forces(pos, z, cell, pbc, di, hp, W)
        lo, hi = int(batch.struct_ptr[b]), int(batch.struct_ptr[b + 1])
        E[b] = o["E"]
        Fo[lo:hi] = o["F"]
    rE = E - np.asarray(E_ref, dtype=np.float64)
    rF = Fo - np.asarray(F_ref, dtype=np.float64).reshape(N, 3)
    loss_E = float(np.mean(np.abs(rE))) if B else 0.0
    loss_F = float(np.mean(np.abs(rF))) if N else 0.0
    c = np.sign(rE) / max(B, 1)
    u = force_weight * np.sign(rF) / max(3 * N, 1)
    grad = {k: np.zeros(np.shape(val)) for k, val in W.items()}
    for b in range(B):
        pos, z, cell, pbc, _ = batch.structure(b)
        lo, hi = int(batch.struct_ptr[b]), int(batch.struct_ptr[b + 1])
        if hi == lo:
            continue
        part = structure_loss_grad_terms(pos, z, cell, pbc, ds[b], hp, W, c[b], u[lo:hi])
        for k in part:
            grad[k] += part[k]
    return dict(loss=loss_E + force_weight * loss_F, loss_E=loss_E, loss_F=loss_F, E=E, F=Fo, grad=grad)


def adamw_step(W, G, state, lr: float, beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
               weight_decay: float = 0.01):
    """One AdamW update of every array of W in place order (returns new
    dicts): state = dict(t, m {name: array}, v {name: array}); t counts the
    steps taken before this one."""
    t = state.get("t", 0) + 1
    m0, v0 = state.get("m", {}), state.get("v", {})
    Wn, mn, vn = {}, {}, {}
    for k, th in W.items():
        g = G[k]
        m = beta1 * m0.get(k, np.zeros_like(th)) + (1.0 - beta1) * g
        v = beta2 * v0.get(k, np.zeros_like(th)) + (1.0 - beta2) * g * g
        mhat = m / (1.0 - beta1 ** t)
        vhat = v / (1.0 - beta2 ** t)
        Wn[k] = th * (1.0 - lr * weight_decay) - lr * mhat / (np.sqrt(vhat) + eps)
        mn[k], vn[k] = m, v
    return Wn, dict(t=t, m=mn, v=vn)
