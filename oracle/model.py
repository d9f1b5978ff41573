"""The DLM forward Phi_theta in its two modes (oracle; test infrastructure only).

Sec. 4.1 of the paper writes Phi_theta(g; C) for the generation forward that
uses prompt cache C, and C_p(g) for the prompt K/V of every layer obtained
when the response is g (App. A.1, Eq. app-cached).

* Eager / full forward (Eq. archer-fresh, Eq. app-eager):
  z*_t = Phi_theta(g_t; C_p(g_t)) -- all P+G positions are recomputed and the
  prompt K/V of every layer is returned as the new cache
  (FullForward of Algorithm 1).
* Cached forward (Eq. archer-cached, Eq. app-cached):
  zhat_t = Phi_theta(g_t; C_p(g_r)) -- only the G response positions are
  recomputed; at every layer their queries attend, with no causal mask, to
  [K_p(g_r) || K_g(g_t)] and [V_p(g_r) || V_g(g_t)] (Eq. archer-attention)
  (CachedForward of Algorithm 1).

The backbone itself is not specified by the paper beyond the model families
it evaluates (LLaDA, Dream, DiffuCoder).  The reading used here: a pre-norm
bidirectional transformer -- x <- E[tok]; per layer
x += Attn(RMSNorm(x)) W_o^T and x += SwiGLU(RMSNorm(x)) W_down^T; final RMSNorm
and an untied LM head; attention scale 1/sqrt(hd); no biases; grouped-query
attention with query head h reading key/value head h // (Hq/Hkv); RoPE at
absolute positions (prompt 0..P-1, response P..P+G-1).  The prompt K is
cached after RoPE (positions never change, so this equals caching it before).

Precision (the paper fixes none).  bf16 models: weights are bf16, and the
oracle rounds exactly where the bf16 path stores values with few bits: the
post-RoPE queries and keys and the values (hence the prompt cache) are
stored as fp16, and the activation operand of every projection named in
``m.single_term`` ("qkv": the normalised attention input, "o": the attention
output, "gateup": the normalised MLP input, "down": the SwiGLU product,
"head": the final normalised hidden state) as a single bf16 value.  The bf16
path carries the other activations, and the attention probabilities, at 16
or more significant bits, so the oracle keeps those unrounded; the residual
stream and the logits are not rounded either.  With ``m.gateup_fp16`` the
gate/up projection multiplies single fp16 operands: its input (the
normalised MLP input) and its two weight matrices are each rounded to fp16
(for the weights, bf16 values, this is exact unless a magnitude lies below
2^-14).  fp32 models round nowhere.
"""

from __future__ import annotations

import numpy as np

from .numerics import attention, linear, rms_norm, rope, round_bf16, round_fp16, silu, weights_f64


def _qkv_store(m, x):
    """Queries, keys and values as the path stores them (fp16 for bf16 models)."""
    return round_fp16(x) if m.dtype == "bf16" else x


def _gateup_fp16(m) -> bool:
    return m.dtype == "bf16" and bool(getattr(m, "gateup_fp16", False))


def _operand(m, name, x):
    """Activation operand of projection ``name``: single bf16 where the model says
    so, a single fp16 value for gate/up under ``gateup_fp16``."""
    if name == "gateup" and _gateup_fp16(m):
        return round_fp16(x)
    single = m.dtype == "bf16" and name in getattr(m, "single_term", ())
    return round_bf16(x) if single else x


def _gateup_weight(m, w):
    """A gate or up matrix as the path multiplies it (fp16 under ``gateup_fp16``)."""
    return round_fp16(weights_f64(w)) if _gateup_fp16(m) else w


def transformer(W: dict, m, tokens: np.ndarray, positions: np.ndarray,
                prefix_kv: list | None = None, out_rows: np.ndarray | None = None,
                keep_hidden: bool = False):
    """Run the bidirectional transformer on ``tokens`` at ``positions``.

    ``prefix_kv`` -- optional per-layer ``(K, V)``, each ``[Hkv][n_prefix][hd]``,
    prepended (in that order) to the keys/values computed from ``tokens`` at
    every layer.  ``out_rows`` -- rows whose logits are returned (default all).

    Returns ``(z, kv, hidden)``: logits ``[len(out_rows)][V]``; per-layer
    ``(K, V)`` of the computed rows, each ``[Hkv][n][hd]`` (post-RoPE, rounded
    like the cache); and, if ``keep_hidden``, the residual stream after the
    embedding and after every layer (``[L+1][n][d]``) plus the final
    normalised hidden state of ``out_rows``.
    """
    tokens = np.asarray(tokens)
    positions = np.asarray(positions)
    n = tokens.shape[0]
    d, hq, hkv, hd = m.d_model, m.n_heads, m.n_kv_heads, m.head_dim
    group = hq // hkv
    if out_rows is None:
        out_rows = np.arange(n)

    x = weights_f64(W["tok_emb"][tokens])
    hidden = [x.copy()] if keep_hidden else None
    kv = []
    for l in range(m.n_layers):
        Wl = W["layers"][l]
        # attention block
        a = _operand(m, "qkv", rms_norm(x, Wl["attn_norm"], m.rms_eps))
        qkv = linear(a, Wl["w_qkv"])
        q = qkv[:, : hq * hd].reshape(n, hq, hd)
        k = qkv[:, hq * hd: (hq + hkv) * hd].reshape(n, hkv, hd)
        v = qkv[:, (hq + hkv) * hd:].reshape(n, hkv, hd)
        q = _qkv_store(m, rope(q, positions, m.rope_theta))
        k = _qkv_store(m, rope(k, positions, m.rope_theta))
        v = _qkv_store(m, v)
        k_rows = k.transpose(1, 0, 2)          # [Hkv][n][hd]
        v_rows = v.transpose(1, 0, 2)
        kv.append((k_rows, v_rows))
        if prefix_kv is not None:
            k_all = np.concatenate([prefix_kv[l][0], k_rows], axis=1)
            v_all = np.concatenate([prefix_kv[l][1], v_rows], axis=1)
        else:
            k_all, v_all = k_rows, v_rows
        o = np.empty((n, hq, hd))
        for h in range(hq):
            o[:, h, :] = attention(q[:, h, :], k_all[h // group], v_all[h // group])
        o = _operand(m, "o", o.reshape(n, hq * hd))
        x = x + linear(o, Wl["w_o"])
        # SwiGLU MLP block
        b = _operand(m, "gateup", rms_norm(x, Wl["mlp_norm"], m.rms_eps))
        gate = linear(b, _gateup_weight(m, Wl["w_gate"]))
        up = linear(b, _gateup_weight(m, Wl["w_up"]))
        hmid = _operand(m, "down", silu(gate) * up)
        x = x + linear(hmid, Wl["w_down"])
        if keep_hidden:
            hidden.append(x.copy())
    c = _operand(m, "head", rms_norm(x[out_rows], W["final_norm"], m.rms_eps))
    z = linear(c, W["lm_head"])
    if keep_hidden:
        return z, kv, (np.stack(hidden), c)
    return z, kv, None


def full_forward(W: dict, m, prompt: np.ndarray, g: np.ndarray, keep_hidden: bool = False):
    """FullForward(p, g): exact logits z* = Phi_theta(g; C_p(g)) and the new cache.

    Recomputes all N = P + G positions of [p; g] (Eq. archer-fresh).  Returns
    ``(z [G][V], cache, hidden)`` where ``cache`` is C_p(g): per layer the
    post-RoPE prompt K and the prompt V, each ``[Hkv][P][hd]``.
    """
    P, G = len(prompt), len(g)
    tokens = np.concatenate([np.asarray(prompt), np.asarray(g)])
    positions = np.arange(P + G)
    z, kv, hidden = transformer(W, m, tokens, positions, None,
                                out_rows=np.arange(P, P + G), keep_hidden=keep_hidden)
    cache = [(k[:, :P, :].copy(), v[:, :P, :].copy()) for (k, v) in kv]
    return z, cache, hidden


def cached_forward(W: dict, m, g: np.ndarray, cache: list, prompt_len: int,
                   keep_hidden: bool = False):
    """CachedForward(g; C_r): zhat = Phi_theta(g; C_r) with C_r = C_p(g_r).

    Only the G response rows are recomputed (at positions P..P+G-1); their
    queries attend to the anchored prompt K/V followed by the fresh response
    K/V at every layer (Eq. archer-attention).  No response tensor from an
    earlier step is used (Prop. app-revisability).
    """
    G = len(g)
    positions = np.arange(prompt_len, prompt_len + G)
    z, _, hidden = transformer(W, m, np.asarray(g), positions, prefix_kv=cache,
                               keep_hidden=keep_hidden)
    return z, hidden
