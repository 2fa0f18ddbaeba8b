"""FP64 PaiNN forces F_i = -dE/dx_i by a hand-written reverse pass (oracle;
test infrastructure only).

The paper's screening throughput counts energies and forces, and its largest
single inference gain comes from computing the force gradient in the same
pass as the energy (section "Optimizing the Inference Pipeline", Fig. 4).
The energy is the model of `oracle.painn`; here its gradient with respect to
the positions is taken by the chain rule, step by step in reverse order.  The
radius graph (and the neighbour cap) is held fixed: it is piecewise constant
in the positions, and the cosine cutoff makes every message vanish with zero
slope at r_c, so the energy is continuously differentiable across an edge
entering or leaving the graph.

Reverse pass, with g_X = dE/dX:
  readout     g_z(last) = 1 per atom; g_y(m) = g_z(m) W_m; g_z(m-1) =
              g_y(m) * silu'(z(m-1))  ->  g_s = g_y(0)
  update      (inputs s, v after the message; U, V, n, a as in the forward)
              g_avv = sum_c g_v[c] U[c];  g_asv = g_s <U, V>;  g_ass = g_s
              g_U[c] = g_v[c] a_vv + g_s a_sv V[c];  g_V[c] = g_s a_sv U[c]
              g_za = (g_a W2a) * silu'(za);  [g_s' ; g_n] = g_za W1a
              g_V[c] += g_n V[c] / n   (taken as 0 where n = 0, the norm's
              subgradient; the forward keeps eps = 0, reading R27)
              g_s <- g_s + g_s';  g_v[c] <- g_v[c] + g_U[c] WU + g_V[c] WV
  message     (edge e: receiver i, sender j; residual paths pass g_s, g_v)
              g_hs_j += g_s_i * w^s;  A_v = sum_c g_v_i[c] v_j[c];
              g_hv_j += A_v * w^v;    A_r = sum_c g_v_i[c] rhat[c];
              g_hr_j += A_r * w^r;    g_v_j[c] += g_v_i[c] * h^v_j * w^v
              g_w = [g_s_i * h^s_j | A_v * h^v_j | A_r * h^r_j]
              g_rhat[c] += sum_f g_v_i[c] h^r_j w^r
              g_d += < g_w , dw/dd >,  dw/dd = f_c'(d)(Wf g + bf) + f_c(d) Wf g'(d)
  phi         g_z1 = (g_h W2) * silu'(z1);  g_s += g_z1 W1
  geometry    g_r = g_d rhat + (g_rhat - (g_rhat . rhat) rhat) / d
              r = x_j - x_i + t:  dE/dx_j += g_r,  dE/dx_i -= g_r

silu'(x) = sig(x) (1 + x (1 - sig(x))), sig the logistic function.
Basis derivatives: Gaussian g_k' = -2 gamma (d - mu_k) g_k; Bessel
g_n' = (n pi / r_c) cos(n pi d / r_c) / d - sin(n pi d / r_c) / d^2;
f_c' = -(pi / (2 r_c)) sin(pi d / r_c).
"""
from __future__ import annotations

import numpy as np

from .neighbors import edge_vectors, radius_graph
from .painn import (RBF_BESSEL, RBF_GAUSSIAN, cosine_cutoff, dense, phi, radial_basis, silu)


def dsilu(x):
    sg = 1.0 / (1.0 + np.exp(-x))
    return sg * (1.0 + x * (1.0 - sg))


def radial_basis_deriv(d, K: int, cutoff: float, rbf_type: int):
    """d g_k / d d for the basis of `oracle.painn.radial_basis`."""
    d = np.asarray(d, dtype=np.float64)
    if rbf_type == RBF_GAUSSIAN:
        delta = cutoff / (K - 1)
        mu = np.arange(K, dtype=np.float64) * delta
        gamma = 1.0 / (2.0 * delta * delta)
        x = d[..., None] - mu
        return -2.0 * gamma * x * np.exp(-gamma * x * x)
    if rbf_type == RBF_BESSEL:
        w = np.arange(1, K + 1, dtype=np.float64) * (np.pi / cutoff)
        dd = d[..., None]
        return w * np.cos(w * dd) / dd - np.sin(w * dd) / (dd * dd)
    raise ValueError(f"unknown radial basis {rbf_type}")


def cosine_cutoff_deriv(d, cutoff: float):
    d = np.asarray(d, dtype=np.float64)
    return np.where(d < cutoff, -0.5 * (np.pi / cutoff) * np.sin(np.pi * d / cutoff), 0.0)


def readout_grad(s, W, hp, dataset_id: int):
    """dE/ds of the per-atom readout summed over atoms: [n, F]."""
    layers = [(W[f"shared{m}.w"], W[f"shared{m}.b"]) for m in range(len(hp.shared_dims))]
    layers += [(W[f"head{dataset_id}.{m}.w"], W[f"head{dataset_id}.{m}.b"])
               for m in range(len(hp.branch_dims))]
    z = []
    y = s
    for m, (w, b) in enumerate(layers):
        zm = dense(y, w, b)
        z.append(zm)
        y = silu(zm) if m < len(layers) - 1 else zm
    g = np.ones((s.shape[0], 1))                  # dE/de_i = 1
    for m in range(len(layers) - 1, -1, -1):
        g = g @ layers[m][0]                      # to the layer's input
        if m > 0:
            g = g * dsilu(z[m - 1])
    return g


def structure_forces(pos, species, cell, pbc, dataset_id, hp, W, head_weights=None):
    """Energy and forces of one structure.  Returns dict(E=float, F=[n, 3],
    n_edges=int).  With `head_weights` (one weight per head, 0 for a skipped
    head) the energy is the blend sum_h w_h E_h of every head over the shared
    final features (section "Composition-conditioned branch weighting"); the
    weights depend on the composition only, so the readout gradient is
    sum_h w_h dE_h/ds."""
    F, K, rc = hp.F, hp.K, hp.cutoff
    z = np.asarray(species)
    x = np.asarray(pos, dtype=np.float64)
    n = len(z)
    recv, send, shift = radius_graph(x, cell, pbc, rc, getattr(hp, "max_neighbors", 0))
    r = edge_vectors(x, cell, recv, send, shift)
    d2 = (r[:, 0] * r[:, 0] + r[:, 1] * r[:, 1]) + r[:, 2] * r[:, 2]
    d = np.sqrt(d2)
    rhat = r / d[:, None]
    g = radial_basis(d, K, rc, hp.rbf_type)
    dg = radial_basis_deriv(d, K, rc, hp.rbf_type)
    fc = cosine_cutoff(d, rc)
    dfc = cosine_cutoff_deriv(d, rc)

    # forward, keeping what the reverse pass reads
    s = W["emb"][z].copy()
    v = np.zeros((n, 3, F))
    saved = []
    for l in range(hp.L):
        h = phi(s, W, l)
        lin = dense(g, W[f"l{l}.filt_w"], W[f"l{l}.filt_b"])       # Wf g + bf
        w = fc[:, None] * lin
        dw = dfc[:, None] * lin + fc[:, None] * (dg @ W[f"l{l}.filt_w"].T)
        hj = h[send]
        ms = hj[:, :F] * w[:, :F]
        mv = (v[send] * (hj[:, None, F:2 * F] * w[:, None, F:2 * F])
              + rhat[:, :, None] * (hj[:, None, 2 * F:] * w[:, None, 2 * F:]))
        s_mid = s.copy()
        v_mid = v.copy()
        np.add.at(s_mid, recv, ms)
        np.add.at(v_mid, recv, mv)
        U = v_mid @ W[f"l{l}.U"].T
        V = v_mid @ W[f"l{l}.V"].T
        nrm = np.sqrt(np.sum(V * V, axis=1))
        za = dense(np.concatenate([s_mid, nrm], axis=1), W[f"l{l}.upd_w1"], W[f"l{l}.upd_b1"])
        a = dense(silu(za), W[f"l{l}.upd_w2"], W[f"l{l}.upd_b2"])
        a_vv, a_sv, a_ss = a[:, :F], a[:, F:2 * F], a[:, 2 * F:]
        UV = np.sum(U * V, axis=1)
        saved.append(dict(s=s, v=v, h=h, w=w, dw=dw, s_mid=s_mid, v_mid=v_mid,
                          U=U, V=V, nrm=nrm, za=za, a_vv=a_vv, a_sv=a_sv))
        v = v_mid + a_vv[:, None, :] * U
        s = s_mid + a_sv * UV + a_ss
    from .painn import readout
    if head_weights is None:
        E = float(np.sum(readout(s, W, hp, dataset_id)))
        gs = readout_grad(s, W, hp, dataset_id)
    else:
        E, gs = 0.0, np.zeros_like(s)
        for h, wh in enumerate(head_weights):
            if wh != 0.0:
                E += wh * float(np.sum(readout(s, W, hp, h)))
                gs = gs + wh * readout_grad(s, W, hp, h)

    # reverse
    gv = np.zeros((n, 3, F))
    gd = np.zeros(len(recv))
    grh = np.zeros((len(recv), 3))
    for l in range(hp.L - 1, -1, -1):
        S = saved[l]
        U, V, nrm, a_vv, a_sv = S["U"], S["V"], S["nrm"], S["a_vv"], S["a_sv"]
        # update block
        g_avv = np.sum(gv * U, axis=1)
        g_asv = gs * np.sum(U * V, axis=1)
        g_a = np.concatenate([g_avv, g_asv, gs], axis=1)
        gU = gv * a_vv[:, None, :] + (gs * a_sv)[:, None, :] * V
        gV = (gs * a_sv)[:, None, :] * U
        g_za = (g_a @ W[f"l{l}.upd_w2"]) * dsilu(S["za"])
        g_in = g_za @ W[f"l{l}.upd_w1"]
        gs = gs + g_in[:, :F]
        g_n = g_in[:, F:]
        safe = np.where(nrm > 0, nrm, 1.0)
        gV = gV + np.where(nrm > 0, g_n / safe, 0.0)[:, None, :] * V
        gv = gv + gU @ W[f"l{l}.U"] + gV @ W[f"l{l}.V"]
        # message (residual paths keep gs, gv)
        h, vv, w, dw = S["h"], S["v"], S["w"], S["dw"]
        gsi, gvi = gs[recv], gv[recv]                # [E, F], [E, 3, F]
        hs, hv, hr = h[send, :F], h[send, F:2 * F], h[send, 2 * F:]
        A_v = np.sum(gvi * vv[send], axis=1)         # [E, F]
        A_r = np.sum(gvi * rhat[:, :, None], axis=1)
        g_h = np.zeros((n, 3 * F))
        np.add.at(g_h, send, np.concatenate([gsi * w[:, :F], A_v * w[:, F:2 * F],
                                             A_r * w[:, 2 * F:]], axis=1))
        gv_new = gv.copy()
        np.add.at(gv_new, send, gvi * (hv * w[:, F:2 * F])[:, None, :])
        g_w = np.concatenate([gsi * hs, A_v * hv, A_r * hr], axis=1)
        gd += np.sum(g_w * dw, axis=1)
        grh += np.sum(gvi * (hr * w[:, 2 * F:])[:, None, :], axis=2)
        # phi
        z1 = dense(S["s"], W[f"l{l}.phi_w1"], W[f"l{l}.phi_b1"])
        g_z1 = (g_h @ W[f"l{l}.phi_w2"]) * dsilu(z1)
        gs = gs + g_z1 @ W[f"l{l}.phi_w1"]
        gv = gv_new
    # geometry
    g_r = gd[:, None] * rhat + (grh - np.sum(grh * rhat, axis=1)[:, None] * rhat) / d[:, None]
    dEdx = np.zeros((n, 3))
    np.add.at(dEdx, send, g_r)
    np.subtract.at(dEdx, recv, g_r)
    return dict(E=E, F=-dEdx, n_edges=len(recv))


def structure_forces_blend(pos, species, cell, pbc, hp, W, skip: float = 0.0):
    """Blended-head energy and forces: the branch-weighting MLP's weights of
    the structure's composition, heads below `skip` left out (not
    renormalised).  Returns dict(E, F, w)."""
    from .painn import blend_weights, composition
    w = blend_weights(composition(species, hp.n_species), hp, W)
    kept = np.where(w >= skip, w, 0.0)
    out = structure_forces(pos, species, cell, pbc, 0, hp, W, head_weights=kept)
    out["w"] = w
    return out


def batch_forces(batch, hp, W, structures=None):
    """Energies [m] and forces (list of [n_b, 3]) of the listed structures."""
    idx = range(batch.n_struct) if structures is None else structures
    E, Fs = [], []
    for b in idx:
        pos, z, cell, pbc, ds = batch.structure(int(b))
        out = structure_forces(pos, z, cell, pbc, ds if hp.n_heads > 1 else 0, hp, W)
        E.append(out["E"])
        Fs.append(out["F"])
    return np.array(E), Fs
