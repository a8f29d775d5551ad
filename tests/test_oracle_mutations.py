"""Plant plausible mistakes in the oracle (on the CPU) and check that a pin catches each.

A mutation replaces one oracle function by a copy carrying one mistake: a dropped
term, a wrong sign or index, a transposed operand, a wrong layout or scale.  The
pins must fail for every one of them, otherwise they would not pin the oracle.
"""
import math

import numpy as np
import pytest

import oracle_pins
from oracle import luna_oracle as O

_orig = {k: getattr(O, k) for k in ("project", "psi", "featuremap", "attn_noncausal", "attn_causal",
                                    "attn_causal_chunked", "kernel_matrix", "psi_pwl", "pwl_tables",
                                    "sufficient_statistics", "attn_quadratic_rows")}


def _psi_mut(kind):
    def psi(u, fc1_w, fc1_b, fc2_w, fc2_b, nonneg=True):
        u = np.asarray(u, float)
        a_all, c_all, f_all, g_all = (np.asarray(x, float) for x in (fc1_w, fc1_b, fc2_w, fc2_b))
        L = f_all.shape[0]
        shared = a_all.shape[0] == 1
        flat = u.reshape(-1)
        out = np.empty((flat.size, L))
        for l in range(L):
            idx = 0 if (shared or kind == "first_layer_of_channel0") else l
            a, c = a_all[idx], c_all[idx]
            if kind == "sign_c":
                c = -c
            hid = np.maximum(flat[:, None] * a[None, :] + c[None, :], 0.0)
            if kind == "no_hidden_relu":
                hid = flat[:, None] * a[None, :] + c[None, :]
            y = hid @ f_all[l] + (0.0 if kind == "drop_g" else g_all[l])
            out[:, l] = (np.maximum(y, 0.0) if (nonneg and kind != "no_output_relu") else y)
        return out.reshape(u.shape + (L,))
    return psi


def _featuremap_mut(kind):
    def featuremap(X, p):
        X = np.asarray(X, float)
        if p.get("per_head", False):
            H = X.shape[-3]
            return np.stack([featuremap(X[..., h, :, :], O._head_params(p, h)) for h in range(H)], axis=-3)
        u = O.project(X, p["W"], p["b"])
        y = O.psi(u, p["fc1_w"], p["fc1_b"], p["fc2_w"], p["fc2_b"], p["nonneg"])
        M, L = y.shape[-2], y.shape[-1]
        if kind == "channel_major":
            y = np.swapaxes(y, -1, -2)
        scale = 1.0 if kind == "no_scale" else 1.0 / math.sqrt(M)
        if kind == "scale_by_M":
            scale = 1.0 / M
        return y.reshape(y.shape[:-2] + (M * L,)) * scale
    return featuremap


def _noncausal_mut(kind):
    def attn_noncausal(Q, K, V, p, eps=1e-6):
        phiQ, phiK = O.featuremap(Q, p), O.featuremap(K, p)
        if kind == "q_for_k":
            phiK = phiQ
        S, z = O.sufficient_statistics(phiK, V)
        num = phiQ @ S
        den = (phiQ @ z[..., :, None])[..., 0]
        if kind == "den_from_q":
            den = phiQ.sum(axis=-1) * phiK.shape[-2]
        if kind == "no_eps":
            eps = 0.0
        return num / (den + eps)[..., None]
    return attn_noncausal


def _causal_mut(kind):
    def attn_causal(Q, K, V, p, eps=1e-6):
        phiQ, phiK, V = O.featuremap(Q, p), O.featuremap(K, p), np.asarray(V, float)
        lead, n, D = phiQ.shape[:-2], phiQ.shape[-2], phiQ.shape[-1]
        S = np.zeros(lead + (D, V.shape[-1]))
        z = np.zeros(lead + (D,))
        out = np.empty(lead + (n, V.shape[-1]))
        for t in range(n):
            if kind != "exclusive":
                S += phiK[..., t, :, None] * V[..., t, None, :]
                z += phiK[..., t, :]
            q = phiQ[..., t, :]
            out[..., t, :] = (q[..., None, :] @ S)[..., 0, :] / ((q * z).sum(-1) + eps)[..., None]
            if kind == "exclusive":
                S += phiK[..., t, :, None] * V[..., t, None, :]
                z += phiK[..., t, :]
        return out
    return attn_causal


def _step_mut(kind):
    def attn_causal_step(Q, K, V, p, S, z, eps=1e-6):
        phiQ, phiK, V = O.featuremap(Q, p), O.featuremap(K, p), np.asarray(V, float)
        S, z = np.array(S, float), np.array(z, float)
        if kind == "drop_prefix":
            S, z = np.zeros_like(S), np.zeros_like(z)
        m = phiQ.shape[-2]
        out = np.empty(phiQ.shape[:-1] + (V.shape[-1],))
        for t in range(m):
            S += phiK[..., t, :, None] * V[..., t, None, :]
            if kind != "stale_z":
                z += phiK[..., t, :]
            q = phiQ[..., t, :]
            out[..., t, :] = (q[..., None, :] @ S)[..., 0, :] / ((q * z).sum(-1) + eps)[..., None]
        return out, S, z
    return attn_causal_step


def _chunked_mut(kind):
    def attn_causal_chunked(Q, K, V, p, chunk, eps=1e-6):
        phiQ, phiK, V = O.featuremap(Q, p), O.featuremap(K, p), np.asarray(V, float)
        lead, n, D = phiQ.shape[:-2], phiQ.shape[-2], phiQ.shape[-1]
        S = np.zeros(lead + (D, V.shape[-1]))
        z = np.zeros(lead + (D,))
        out = np.empty(lead + (n, V.shape[-1]))
        for s0 in range(0, n, chunk):
            s1 = min(n, s0 + chunk)
            q, k, v = phiQ[..., s0:s1, :], phiK[..., s0:s1, :], V[..., s0:s1, :]
            P = np.tril(q @ np.swapaxes(k, -1, -2), -1 if kind == "strict_tril" else 0)
            num = P @ v + q @ S
            den = P.sum(-1) + (q @ z[..., :, None])[..., 0]
            if kind == "no_carry_den":
                den = P.sum(-1)
            out[..., s0:s1, :] = num / (den + eps)[..., None]
            S = S + np.swapaxes(k, -1, -2) @ v
            z = z + k.sum(-2)
        return out
    return attn_causal_chunked


def _project_mut(kind):
    def project(X, W, b):
        X, W, b = (np.asarray(x, float) for x in (X, W, b))
        if kind == "no_bias":
            return X @ W.T
        if kind == "transposed_W":
            return X @ W.reshape(W.shape[::-1]) + b
        return X @ W.T - b
    return project


def _kernel_mut(kind):
    def kernel_matrix(Xq, Xk, p):
        return _orig["kernel_matrix"](Xq, Xk, p) * (p["W"].shape[-2] if kind == "no_average" else 1.0) + (
            1e-3 if kind == "offset" else 0.0)
    return kernel_matrix


def _pwl_mut(kind):
    def psi_pwl(u, tables, nonneg=True):
        bp, s, t = tables
        u = np.asarray(u, float)
        j = np.searchsorted(bp, u, side="left")
        j = np.minimum(j + 1, len(bp)) if kind == "segment_plus_one" else j
        y = s[j] * u[..., None] + t[j]
        return np.maximum(y, 0.0) if nonneg else y
    return psi_pwl


MUTATIONS = {
    "psi_drop_g": ("psi", _psi_mut("drop_g")),
    "psi_sign_c": ("psi", _psi_mut("sign_c")),
    "psi_no_output_relu": ("psi", _psi_mut("no_output_relu")),
    "psi_no_hidden_relu": ("psi", _psi_mut("no_hidden_relu")),
    "psi_wrong_channel_first_layer": ("psi", _psi_mut("first_layer_of_channel0")),
    "featuremap_channel_major": ("featuremap", _featuremap_mut("channel_major")),
    "featuremap_no_scale": ("featuremap", _featuremap_mut("no_scale")),
    "featuremap_scale_by_M": ("featuremap", _featuremap_mut("scale_by_M")),
    "project_no_bias": ("project", _project_mut("no_bias")),
    "project_transposed_W": ("project", _project_mut("transposed_W")),
    "project_bias_sign": ("project", _project_mut("bias_sign")),
    "noncausal_q_for_k": ("attn_noncausal", _noncausal_mut("q_for_k")),
    "noncausal_den_from_q": ("attn_noncausal", _noncausal_mut("den_from_q")),
    "noncausal_no_eps": ("attn_noncausal", _noncausal_mut("no_eps")),
    "causal_exclusive_prefix": ("attn_causal", _causal_mut("exclusive")),
    "chunked_strict_tril": ("attn_causal_chunked", _chunked_mut("strict_tril")),
    "step_drops_prefix": ("attn_causal_step", _step_mut("drop_prefix")),
    "step_stale_z": ("attn_causal_step", _step_mut("stale_z")),
    "chunked_no_carry_den": ("attn_causal_chunked", _chunked_mut("no_carry_den")),
    "kernel_no_average": ("kernel_matrix", _kernel_mut("no_average")),
    "kernel_offset": ("kernel_matrix", _kernel_mut("offset")),
    "pwl_segment_plus_one": ("psi_pwl", _pwl_mut("segment_plus_one")),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(O, attr, fn)
    failed = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(O)
        except Exception:
            failed.append(pin.__name__)
    assert failed, f"no pin catches the planted mistake {name}"
