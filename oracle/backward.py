"""Plain CPU oracle of the gradients of event-factorized attention over
whole branches (the training form of the §3.4 mask: query token j of branch
e sees every prefix token and its own rows 0 .. min(j, n_e - 1)).

TEST INFRASTRUCTURE ONLY: imported by the test suite, never by the library;
it shares nothing with it.

Given the forward pass's output O and log-normalisers lse (as the forward
returned them) and the gradient dO of a loss with respect to O, for every
live query row i (stream e with n_e > 0, token j, head h of kv head
g = h // G) over its visible keys k:
    p_ik  = exp(tau <q_i, k_k> - lse_i)            (the attention weights)
    D_i   = <dO_i, O_i>
    ds_ik = p_ik (<dO_i, v_k> - D_i)
    dq_i  = tau sum_k ds_ik k_k
    dk_k += tau ds_ik q_i,      dv_k += p_ik dO_i.
That is the chain rule through O_i = sum_k p_ik v_k with p the softmax of
tau <q_i, k>: with O and lse exact it is the gradient of sum_i <dO_i, O_i>.
Readings: rows of ended streams (n_e <= 0) have no output, so they add
nothing and their dq is 0; keys nobody sees (cache rows at or past n_e)
get zero gradients; tau is 1/sqrt(D) unless given.

Arithmetic in float64; bf16 inputs (uint16 bit patterns) are widened
exactly.
"""
from __future__ import annotations

import numpy as np


def _widen(a) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def attn_prefill_backward(q, k_prefix, v_prefix, k_event, v_event, event_lens, out, lse, dout, scale: float = 0.0):
    """One video: q, out, dout [E, N, H_q, D]; k/v_prefix [L, H_kv, D];
    k/v_event [E, cap, H_kv, D]; lse [E, N, H_q].  Returns (dq, dk_prefix,
    dv_prefix, dk_event, dv_event), float64, shaped like their inputs."""
    q, kp, vp, ke, ve = (_widen(x) for x in (q, k_prefix, v_prefix, k_event, v_event))
    out, dout = _widen(out), _widen(dout)
    lse = np.asarray(lse, dtype=np.float64)
    n = np.asarray(event_lens, dtype=np.int64)
    E, N, H_q, D = q.shape
    L, H_kv = kp.shape[0], kp.shape[1]
    G = H_q // H_kv
    tau = scale if scale > 0 else 1.0 / np.sqrt(D)
    dq = np.zeros_like(q)
    dkp, dvp = np.zeros_like(kp), np.zeros_like(vp)
    dke, dve = np.zeros_like(ke), np.zeros_like(ve)
    for e in range(E):
        if n[e] <= 0:
            continue
        for j in range(N):
            own = min(j, n[e] - 1) + 1  # own rows 0 .. min(j, n_e - 1)
            for h in range(H_q):
                g = h // G
                keys = np.concatenate([kp[:, g], ke[e, :own, g]])
                vals = np.concatenate([vp[:, g], ve[e, :own, g]])
                p = np.exp(tau * (keys @ q[e, j, h]) - lse[e, j, h])
                do = dout[e, j, h]
                ds = p * (vals @ do - do @ out[e, j, h])
                dq[e, j, h] = tau * (ds @ keys)
                dkp[:, g] += tau * ds[:L, None] * q[e, j, h]
                dke[e, :own, g] += tau * ds[L:, None] * q[e, j, h]
                dvp[:, g] += p[:L, None] * do
                dve[e, :own, g] += p[L:, None] * do
    return dq, dkp, dvp, dke, dve


def sampled_gradients(q, k_prefix, v_prefix, k_event, v_event, event_lens, out, lse, dout,
                      rows=(), prefix_keys=(), own_keys=(), scale: float = 0.0):
    """Selected entries of the same gradients, each formed on its own from
    the definitions above, for shapes where the full loop is too slow:
      rows        (e, j, h): dq of that query row over its visible keys;
      prefix_keys (l, g):    dk, dv of prefix row l of kv head g, summed over
                             every live query row of the heads of group g;
      own_keys    (e, t, g): dk, dv of row t of stream e's cache, summed over
                             the rows of stream e whose token j sees it
                             (t < n_e and t <= j).
    Returns (list of dq [D], list of (dk [D], dv [D]) per prefix key, the same
    per own key), float64."""
    q, kp, vp, ke, ve = (_widen(x) for x in (q, k_prefix, v_prefix, k_event, v_event))
    out, dout = _widen(out), _widen(dout)
    lse = np.asarray(lse, dtype=np.float64)
    n = np.asarray(event_lens, dtype=np.int64)
    E, N, H_q, D = q.shape
    H_kv = kp.shape[1]
    G = H_q // H_kv
    tau = scale if scale > 0 else 1.0 / np.sqrt(D)

    dqs = []
    for e, j, h in rows:
        if n[e] <= 0:
            dqs.append(np.zeros(D))
            continue
        g, own = h // G, min(j, n[e] - 1) + 1
        keys = np.concatenate([kp[:, g], ke[e, :own, g]])
        vals = np.concatenate([vp[:, g], ve[e, :own, g]])
        p = np.exp(tau * (keys @ q[e, j, h]) - lse[e, j, h])
        ds = p * (vals @ dout[e, j, h] - dout[e, j, h] @ out[e, j, h])
        dqs.append(tau * (ds @ keys))

    def key_grads(k, v, qs, dos, outs, lses):
        # qs, dos, outs [rows, D], lses [rows]: the query rows that see key k
        p = np.exp(tau * (qs @ k) - lses)
        ds = p * (dos @ v - np.einsum("rd,rd->r", dos, outs))
        return tau * (ds @ qs), p @ dos

    live = n > 0
    pks = []
    for l, g in prefix_keys:
        sl = (live, slice(None), slice(g * G, (g + 1) * G))
        pks.append(key_grads(kp[l, g], vp[l, g], q[sl].reshape(-1, D), dout[sl].reshape(-1, D),
                             out[sl].reshape(-1, D), lse[sl].reshape(-1)))
    oks = []
    for e, t, g in own_keys:
        if t >= n[e]:
            oks.append((np.zeros(D), np.zeros(D)))
            continue
        sl = (e, slice(t, N), slice(g * G, (g + 1) * G))
        oks.append(key_grads(ke[e, t, g], ve[e, t, g], q[sl].reshape(-1, D), dout[sl].reshape(-1, D),
                             out[sl].reshape(-1, D), lse[sl].reshape(-1)))
    return dqs, pks, oks
