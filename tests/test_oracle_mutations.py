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
                                    "sufficient_statistics", "attn_quadratic_rows", "_psi_backward",
                                    "featuremap_backward", "attn_noncausal_backward", "attn_causal_backward")}


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


def _psi_backward_mut(kind):
    def _psi_backward(u, dpsi, fc1_w, fc1_b, fc2_w, fc2_b, nonneg=True):
        u = np.asarray(u, float)
        a_all, c_all, f_all, g_all = (np.asarray(x, float) for x in (fc1_w, fc1_b, fc2_w, fc2_b))
        L = f_all.shape[0]
        shared = a_all.shape[0] == 1
        du = np.zeros(u.shape)
        d1w, d1b, d2w, d2b = (np.zeros(x.shape) for x in (a_all, c_all, f_all, g_all))
        for l in range(L):
            i = 0 if shared else l
            pre = u[:, None] * a_all[i] + c_all[i]
            hid = np.maximum(pre, 0.0)
            y = hid @ f_all[l] + g_all[l]
            mask = (y > 0.0) if (nonneg and kind != "no_output_mask") else 1.0
            dy = dpsi[:, l] * mask
            d2w[l] += hid.T @ dy
            d2b[l] += dy.sum()
            gate = (pre >= 0.0) if kind == "relu_at_zero_passes" else (pre > 0.0)
            dpre = (dy[:, None] * f_all[l]) * gate
            d1w[i] += (dpre * u[:, None]).sum(axis=0) * (0.0 if kind == "drop_dfc1_w" else 1.0)
            d1b[i] += dpre.sum(axis=0)
            du += dpre @ a_all[i]
        return du, d1w, d1b, d2w, d2b
    return _psi_backward


def _fm_backward_mut(kind):
    def featuremap_backward(X, p, dphi):
        dX, g = _orig["featuremap_backward"](X, p, dphi)
        if kind == "scale_missing":
            M = np.shape(p["W"])[-2]
            dX, g = dX * math.sqrt(M), {k: v * math.sqrt(M) for k, v in g.items()}
        if kind == "dW_no_bias_grad":
            g = dict(g)
            g["b"] = np.zeros_like(g["b"])
        return dX, g
    return featuremap_backward


def _nc_backward_mut(kind):
    def attn_noncausal_backward(Q, K, V, p, dO, eps=1e-6):
        V, dO = np.asarray(V, float), np.asarray(dO, float)
        phiQ, phiK = O.featuremap(Q, p), O.featuremap(K, p)
        S, z = O.sufficient_statistics(phiK, V)
        num = phiQ @ S
        den = (phiQ @ z[..., :, None])[..., 0] + eps
        dnum = dO / den[..., None]
        dden = -(dO * num).sum(-1) / den ** 2 * (0.0 if kind == "drop_dden" else 1.0)
        dphiQ = dnum @ np.swapaxes(S, -1, -2) + dden[..., None] * z[..., None, :]
        dS = np.swapaxes(phiQ, -1, -2) @ dnum
        dz = (np.swapaxes(phiQ, -1, -2) @ dden[..., None])[..., 0]
        dphiK = V @ np.swapaxes(dS, -1, -2) + (0.0 if kind == "dphik_no_dz" else dz[..., None, :])
        dV = (phiQ if kind == "dv_from_q" else phiK) @ dS
        dQ, gq = O.featuremap_backward(Q, p, dphiQ)
        dK, gk = O.featuremap_backward(K, p, dphiK)
        return dQ, dK, dV, {k: gq[k] + gk[k] for k in gq}
    return attn_noncausal_backward


def _cs_backward_mut(kind):
    def attn_causal_backward(Q, K, V, p, dO, eps=1e-6):
        if kind == "as_noncausal":
            return _orig["attn_noncausal_backward"](Q, K, V, p, dO, eps)
        V, dO = np.asarray(V, float), np.asarray(dO, float)
        phiQ, phiK = O.featuremap(Q, p), O.featuremap(K, p)
        lead, n, D = phiQ.shape[:-2], phiQ.shape[-2], phiQ.shape[-1]
        S, z = np.zeros(lead + (D, V.shape[-1])), np.zeros(lead + (D,))
        dnum, dden = np.empty(lead + (n, V.shape[-1])), np.empty(lead + (n,))
        dphiQ = np.empty(phiQ.shape)
        for t in range(n):
            S += phiK[..., t, :, None] * V[..., t, None, :]
            z += phiK[..., t, :]
            q = phiQ[..., t, :]
            num = (q[..., None, :] @ S)[..., 0, :]
            den = (q * z).sum(-1) + eps
            dnum[..., t, :] = dO[..., t, :] / den[..., None]
            dden[..., t] = -(dO[..., t, :] * num).sum(-1) / den ** 2
            dphiQ[..., t, :] = (S @ dnum[..., t, :, None])[..., 0] + z * dden[..., t, None]
        dS, dz = np.zeros(S.shape), np.zeros(z.shape)
        dphiK, dV = np.empty(phiK.shape), np.empty(V.shape)
        order = range(n) if kind == "prefix_for_keys" else range(n - 1, -1, -1)
        for t in order:
            if kind != "exclusive_suffix":
                dS += phiQ[..., t, :, None] * dnum[..., t, None, :]
                dz += phiQ[..., t, :] * dden[..., t, None]
            dphiK[..., t, :] = (dS @ V[..., t, :, None])[..., 0] + dz
            dV[..., t, :] = (phiK[..., t, None, :] @ dS)[..., 0, :]
            if kind == "exclusive_suffix":
                dS += phiQ[..., t, :, None] * dnum[..., t, None, :]
                dz += phiQ[..., t, :] * dden[..., t, None]
        dQ, gq = O.featuremap_backward(Q, p, dphiQ)
        dK, gk = O.featuremap_backward(K, p, dphiK)
        return dQ, dK, dV, {k: gq[k] + gk[k] for k in gq}
    return attn_causal_backward


MUTATIONS = {
    "bwd_psi_relu_at_zero_passes": ("_psi_backward", _psi_backward_mut("relu_at_zero_passes")),
    "bwd_psi_no_output_mask": ("_psi_backward", _psi_backward_mut("no_output_mask")),
    "bwd_psi_drop_dfc1_w": ("_psi_backward", _psi_backward_mut("drop_dfc1_w")),
    "bwd_featuremap_scale_missing": ("featuremap_backward", _fm_backward_mut("scale_missing")),
    "bwd_featuremap_no_bias_grad": ("featuremap_backward", _fm_backward_mut("dW_no_bias_grad")),
    "bwd_noncausal_drop_dden": ("attn_noncausal_backward", _nc_backward_mut("drop_dden")),
    "bwd_noncausal_dphik_no_dz": ("attn_noncausal_backward", _nc_backward_mut("dphik_no_dz")),
    "bwd_noncausal_dv_from_q": ("attn_noncausal_backward", _nc_backward_mut("dv_from_q")),
    "bwd_causal_as_noncausal": ("attn_causal_backward", _cs_backward_mut("as_noncausal")),
    "bwd_causal_prefix_for_keys": ("attn_causal_backward", _cs_backward_mut("prefix_for_keys")),
    "bwd_causal_exclusive_suffix": ("attn_causal_backward", _cs_backward_mut("exclusive_suffix")),
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


# ---------------------------------------------------------------------------
# feature-map variants: mistakes planted in oracle/luna_variants.py
# ---------------------------------------------------------------------------

import oracle_variant_pins  # noqa: E402
from oracle import luna_variants as VAR  # noqa: E402

_vorig = {k: getattr(VAR, k) for k in ("rff_cos", "rff_sincos", "performer", "_act", "ch_rms", "mlp_variant",
                                        "attn_from_features", "_mlp_channels")}


def _rff_cos_mut(kind):
    def rff_cos(X, p):
        if p.get("per_head", False):
            return VAR._per_head(rff_cos, np.asarray(X, float), p)
        u = np.asarray(X, float) @ np.asarray(p["W"], float).T + (0.0 if kind == "no_phase" else np.asarray(p["b"]))
        scale = 1.0 / math.sqrt(u.shape[-1]) if kind == "no_sqrt2" else math.sqrt(2.0 / u.shape[-1])
        return scale * (np.sin(u) if kind == "sin" else np.cos(u))
    return rff_cos


def _sincos_mut(kind):
    def rff_sincos(X, p):
        if p.get("per_head", False):
            return VAR._per_head(rff_sincos, np.asarray(X, float), p)
        u = np.asarray(X, float) @ np.asarray(p["W"], float).T + np.asarray(p["b"])
        M = u.shape[-1]
        pair = [np.cos(u), np.sin(u)] if kind == "cos_first" else [np.sin(u), np.cos(u)]
        y = np.stack(pair, axis=-2 if kind == "channel_major" else -1)
        return y.reshape(u.shape[:-1] + (2 * M,)) / math.sqrt(M)
    return rff_sincos


def _performer_mut(kind):
    def performer(X, p):
        X = np.asarray(X, float)
        if p.get("per_head", False):
            return VAR._per_head(performer, X, p)
        d = X.shape[-1]
        u = X @ np.asarray(p["W"], float).T + np.asarray(p["b"])
        sq = (X * X).sum(axis=-1, keepdims=True)
        denom = 2.0 * d if kind == "d_not_sqrt_d" else 2.0 * math.sqrt(d)
        if kind == "plus_norm":
            return np.exp(u + sq / denom) / math.sqrt(u.shape[-1])
        return np.exp(u - sq / denom) / math.sqrt(u.shape[-1])
    return performer


def _act_mut(kind):
    def act(name, z):
        if name == "gelu" and kind == "gelu_as_silu":
            return z / (1.0 + np.exp(-z))
        if name == "silu" and kind == "silu_no_z":
            return 1.0 / (1.0 + np.exp(-z))
        return _vorig["_act"](name, z)
    return act


def _chrms_mut(kind):
    def ch_rms(y, target, eps=1e-6):
        y = np.asarray(y, float)
        L = y.shape[-1]
        if kind == "per_token":
            rms = np.sqrt((y ** 2).mean(axis=-2, keepdims=True) + eps)
        else:
            rms = np.sqrt((y.reshape(-1, L) ** 2).mean(axis=0) + eps)
        s = target / (rms + eps) if kind == "no_clamp" else np.minimum(target / (rms + eps), 1.0)
        return y * s
    return ch_rms


def _mlp_channels_mut(kind):
    def _mlp_channels(X, p):
        u = X @ np.asarray(p["W"], float).T + np.asarray(p["b"])
        y = VAR.psi_act(u, p["fc1_w"], p["fc1_b"], p["fc2_w"], p["fc2_b"], p["nonneg"], p.get("act", "relu"))
        if p.get("env_w") is not None:
            z = X @ np.asarray(p["env_w"], float).T + np.asarray(p["env_b"])
            env = 1.0 / (1.0 + np.exp(z if kind == "env_sign" else -z))
            if kind == "env_on_projection":  # the first L projections gated instead of the channels
                y = y * env[..., :, None][..., : y.shape[-2], :] if env.shape[-1] >= y.shape[-2] else y * env[..., None, :] ** 2
            else:
                y = y * env[..., None, :]
        return y
    return _mlp_channels


def _bank_mut(kind):
    def mlp_variant(X, p):
        if p.get("bank") is None:
            return _vorig["mlp_variant"](X, p)
        X = np.asarray(X, float)
        y = VAR._per_head(VAR._mlp_channels, X, p)
        M, L = y.shape[-2], y.shape[-1]
        w = np.asarray(p["bank"], float)
        if kind == "reversed":
            w = w[::-1]
        out = y @ w
        return out / (M if kind == "scale_by_M" else math.sqrt(M))
    return mlp_variant


def _from_features_mut(kind):
    def attn_from_features(phiQ, phiK, V, eps=1e-6, causal=False):
        if kind == "causal_exclusive" and causal:
            phiQ, phiK, V = (np.asarray(a, float) for a in (phiQ, phiK, V))
            n = phiQ.shape[-2]
            A = np.tril(phiQ @ np.swapaxes(phiK, -1, -2), -1)
            return (A @ V) / (A.sum(-1) + eps)[..., None]
        if kind == "no_normaliser" and not causal:
            phiQ, phiK, V = (np.asarray(a, float) for a in (phiQ, phiK, V))
            return phiQ @ (np.swapaxes(phiK, -1, -2) @ V)
        return _vorig["attn_from_features"](phiQ, phiK, V, eps, causal)
    return attn_from_features


VARIANT_MUTATIONS = {
    "rff_cos_as_sin": ("rff_cos", _rff_cos_mut("sin")),
    "rff_cos_no_sqrt2": ("rff_cos", _rff_cos_mut("no_sqrt2")),
    "rff_cos_no_phase": ("rff_cos", _rff_cos_mut("no_phase")),
    "sincos_cos_first": ("rff_sincos", _sincos_mut("cos_first")),
    "sincos_channel_major": ("rff_sincos", _sincos_mut("channel_major")),
    "performer_norm_over_d": ("performer", _performer_mut("d_not_sqrt_d")),
    "performer_norm_sign": ("performer", _performer_mut("plus_norm")),
    "gelu_as_silu": ("_act", _act_mut("gelu_as_silu")),
    "silu_without_z": ("_act", _act_mut("silu_no_z")),
    "ch_rms_per_token": ("ch_rms", _chrms_mut("per_token")),
    "ch_rms_no_clamp": ("ch_rms", _chrms_mut("no_clamp")),
    "envelope_sign": ("_mlp_channels", _mlp_channels_mut("env_sign")),
    "bank_reversed": ("mlp_variant", _bank_mut("reversed")),
    "bank_scale_by_M": ("mlp_variant", _bank_mut("scale_by_M")),
    "from_features_exclusive_prefix": ("attn_from_features", _from_features_mut("causal_exclusive")),
    "from_features_no_normaliser": ("attn_from_features", _from_features_mut("no_normaliser")),
}


@pytest.mark.parametrize("name", sorted(VARIANT_MUTATIONS))
def test_variant_mutation_is_caught(name, monkeypatch):
    attr, fn = VARIANT_MUTATIONS[name]
    monkeypatch.setattr(VAR, attr, fn)
    failed = []
    for pin in oracle_variant_pins.ALL_PINS:
        try:
            pin(VAR)
        except Exception:
            failed.append(pin.__name__)
    assert failed, f"no pin catches the planted mistake {name}"


# ---------------------------------------------------------------------------
# distillation oracle
# ---------------------------------------------------------------------------
import oracle_distill_pins  # noqa: E402
from oracle import luna_distill as DIS  # noqa: E402

_dorig = {k: getattr(DIS, k) for k in ("teacher", "student", "distill_feature_grads", "distill_backward")}


def _teacher_mut(kind):
    def teacher(Q, K, causal=False):
        Q, K = np.asarray(Q, float), np.asarray(K, float)
        n, d = Q.shape[-2], Q.shape[-1]
        logits = Q @ np.swapaxes(K, -1, -2)
        if kind != "no_scale":
            logits = logits / math.sqrt(d)
        vis = np.tril(np.ones((n, n), bool)) if (causal and kind != "no_mask") else np.ones((n, n), bool)
        logits = np.where(vis, logits, -np.inf)
        e = np.where(vis, np.exp(logits - logits.max(-1, keepdims=True)), 0.0)
        return e / e.sum(-1, keepdims=True)
    return teacher


def _student_mut(kind):
    def student(phiQ, phiK, causal=False, eps=1e-6):
        phiQ, phiK = np.asarray(phiQ, float), np.asarray(phiK, float)
        n = phiQ.shape[-2]
        vis = np.tril(np.ones((n, n), bool)) if causal else np.ones((n, n), bool)
        P = phiQ @ np.swapaxes(phiK, -1, -2)
        den = (P if kind == "den_all_keys" else np.where(vis, P, 0.0)).sum(-1, keepdims=True)
        P = np.where(vis, P, 0.0)
        nt = vis.sum(-1, keepdims=True).astype(float)
        smooth = eps if kind == "eps_not_over_nt" else eps / nt
        return np.where(vis, (P + smooth) / (den + eps), 0.0)
    return student


def _dgrad_mut(kind):
    def distill_feature_grads(Q, K, phiQ, phiK, causal=False, eps=1e-6):
        gq, gk = _dorig["distill_feature_grads"](Q, K, phiQ, phiK, causal, eps)
        phiQ, phiK = np.asarray(phiQ, float), np.asarray(phiK, float)
        if kind == "sign":
            return -gq, -gk
        if kind == "sum_not_mean":
            rows = float(np.prod(np.shape(phiQ)[:-1]))
            return gq * rows, gk * rows
        if kind == "k_untransposed":  # dphi(K) = G phi(Q) instead of G^T phi(Q)
            A = DIS.teacher(Q, K, causal)
            n = A.shape[-1]
            vis = np.tril(np.ones((n, n), bool)) if causal else np.ones((n, n), bool)
            P = np.where(vis, phiQ @ np.swapaxes(phiK, -1, -2), 0.0)
            den = P.sum(-1, keepdims=True)
            nt = vis.sum(-1, keepdims=True).astype(float)
            G = np.where(vis, (1.0 / (den + eps) - A / (P + eps / nt)) / float(np.prod(A.shape[:-1])), 0.0)
            return gq, G @ phiQ
        if kind == "no_den_term":
            A = DIS.teacher(Q, K, causal)
            n = A.shape[-1]
            vis = np.tril(np.ones((n, n), bool)) if causal else np.ones((n, n), bool)
            P = np.where(vis, phiQ @ np.swapaxes(phiK, -1, -2), 0.0)
            nt = vis.sum(-1, keepdims=True).astype(float)
            G = np.where(vis, (-A / (P + eps / nt)) / float(np.prod(A.shape[:-1])), 0.0)
            return G @ phiK, np.swapaxes(G, -1, -2) @ phiQ
        return gq, gk
    return distill_feature_grads


def _dback_mut(kind):
    def distill_backward(Q, K, p, causal=False, eps=1e-6):
        phiQ, phiK = O.featuremap(Q, p), O.featuremap(K, p)
        rows = DIS.distill_rows_features(Q, K, phiQ, phiK, causal, eps)
        dq, dk = DIS.distill_feature_grads(Q, K, phiQ, phiK, causal, eps)
        _, gq = O.featuremap_backward(Q, p, dq)
        _, gk = O.featuremap_backward(K, p, dk)
        if kind == "queries_only":
            return rows, gq
        return rows, {k: gq[k] + gk[k] for k in O.PARAM_NAMES}
    return distill_backward


DISTILL_MUTATIONS = {
    "teacher_without_scale": ("teacher", _teacher_mut("no_scale")),
    "teacher_without_causal_mask": ("teacher", _teacher_mut("no_mask")),
    "student_den_over_all_keys": ("student", _student_mut("den_all_keys")),
    "student_eps_not_over_nt": ("student", _student_mut("eps_not_over_nt")),
    "grads_sign": ("distill_feature_grads", _dgrad_mut("sign")),
    "grads_sum_not_mean": ("distill_feature_grads", _dgrad_mut("sum_not_mean")),
    "grads_key_side_untransposed": ("distill_feature_grads", _dgrad_mut("k_untransposed")),
    "grads_without_den_term": ("distill_feature_grads", _dgrad_mut("no_den_term")),
    "backward_queries_only": ("distill_backward", _dback_mut("queries_only")),
}


@pytest.mark.parametrize("name", sorted(DISTILL_MUTATIONS))
def test_distill_mutation_is_caught(name, monkeypatch):
    attr, fn = DISTILL_MUTATIONS[name]
    monkeypatch.setattr(DIS, attr, fn)
    failed = []
    for pin in oracle_distill_pins.ALL_PINS:
        try:
            pin(DIS)
        except Exception:
            failed.append(pin.__name__)
    assert failed, f"no pin catches the planted mistake {name}"
