"""The paper's unfused formulations and the interlaced gate/up layout, in fp64.

Test infrastructure only (see the package header). The paper states that its
fused attention (GKVC + TPSFLAT, Alg. 3) and fused MLP (Alg. 4) keep the
computation exact (Section 3, opening). These functions compute the same
layer the unfused way so the CPU tests can check that claim on the fp64
oracle:

  * attention_alg1 -- Alg. 1: RoPE, Transpose, Concat of the new K/V after
    the cached rows (a reloading append), then QK^T, Softmax, PV as separate
    whole-tensor operators;
  * mlp_alg2       -- Alg. 2: gate, SiLU, up, elementwise multiply, down;
  * interlace_gate_up / mlp_interlaced -- Alg. 4 with Eq. 29-32: W_gate and
    W_up split along K into half tiles and alternated into one W_gu, one
    projection through W_gu, then siLu_Mul on each tile's halves.

Parity: pinned by equivalence with ``ref`` (checked to 1e-12 relative) and,
through ``ref``, by brute force and the invariants listed there.
"""
from __future__ import annotations

import numpy as np

from . import ref


def attention_alg1(q, k, v, k_cache_bits, v_cache_bits, pos, rope_base, n_kv_heads):
    """Standard attention of Alg. 1 for one sequence.

    q [H, d], k and v [H_kv, d] (as the QKV projection gives them, un-roped);
    caches [H_kv, N_max, d] bf16 bits with N_p = pos valid rows.
    Returns (O [H, d], K_cache' [H_kv, pos+1, d] bits, V_cache' bits).
    """
    H, d = q.shape
    group = H // n_kv_heads
    # Step 1: RoPE on Q and K
    q_rope = ref.rope(q, pos, rope_base)
    k_rope = ref.rope(k, pos, rope_base)
    # Step 2: Transpose [N, H, d] -> [H, N, d] (N = 1)
    q_t = np.transpose(q_rope[None], (1, 0, 2))
    k_t = np.transpose(ref.f64_to_bf16_bits(k_rope)[None], (1, 0, 2))
    v_t = np.transpose(ref.f64_to_bf16_bits(v)[None], (1, 0, 2))
    # Step 3: Concat the cached rows with the new one (reads and rewrites the cache)
    k_cat = np.concatenate([k_cache_bits[:, :pos, :], k_t], axis=1)
    v_cat = np.concatenate([v_cache_bits[:, :pos, :], v_t], axis=1)
    kf = ref.bf16_bits_to_f64(k_cat)
    vf = ref.bf16_bits_to_f64(v_cat)
    # GQA: broadcast each KV head to its group of query heads
    kf = np.repeat(kf, group, axis=0)
    vf = np.repeat(vf, group, axis=0)
    # Step 4: S = Q K^T / sqrt(d)  -> [H, 1, N_t]
    s = np.matmul(q_t, np.transpose(kf, (0, 2, 1))) / np.sqrt(float(d))
    # Step 5: P = softmax(S)
    p = ref.softmax(s)
    # Step 6: O = P V -> [H, 1, d]
    o = np.matmul(p, vf)
    return o[:, 0, :], k_cat, v_cat


def mlp_alg2(h, w_gate, w_up, w_down):
    """Standard MLP of Alg. 2 (five separate operators)."""
    h_g = w_gate @ h            # Step 1
    h_s = ref.silu(h_g)         # Step 2
    h_u = w_up @ h              # Step 3
    h_p = h_u * h_s             # Step 4
    return w_down @ h_p         # Step 5


def interlace_gate_up(w_gate: np.ndarray, w_up: np.ndarray, tile: int) -> np.ndarray:
    """Interlaced W_gu (Alg. 4 input; Section 3.2, item 1).

    With weights stored [out, in] = [K, D], output rows of gate and up are cut
    into tiles of ``tile`` rows; packed block i is [gate rows of tile i; up rows
    of tile i] (Eq. 31: first half gate, second half up). The last tile may be
    shorter when tile does not divide K.
    """
    K, D = w_gate.shape
    blocks = []
    for k0 in range(0, K, tile):
        k1 = min(K, k0 + tile)
        blocks.append(w_gate[k0:k1])
        blocks.append(w_up[k0:k1])
    return np.concatenate(blocks, axis=0)


def mlp_interlaced(h, w_gu: np.ndarray, w_down: np.ndarray, tile: int):
    """Fusion MLP of Alg. 4: one projection through W_gu, siLu_Mul per tile, then down.

    Eq. 29: h_gu = W_gu h; Eq. 30-31: per tile, siLu(gate half) * up half -> h_sm;
    Eq. 32: O = W_down h_sm. Returns (O, h_sm).
    """
    h_gu = w_gu @ h
    K = w_down.shape[1]
    h_sm = np.empty(K)
    r = 0
    for k0 in range(0, K, tile):
        t = min(K, k0 + tile) - k0
        gate_half = h_gu[r:r + t]
        up_half = h_gu[r + t:r + 2 * t]
        h_sm[k0:k0 + t] = ref.silu(gate_half) * up_half
        r += 2 * t
    return w_down @ h_sm, h_sm


def decode_layer_unfused(x_bits, pos, k_cache_bits, v_cache_bits, weights, *, n_heads,
                         n_kv_heads, rope_base, rms_eps, tile=16):
    """The whole layer through Alg. 1 attention and the interlaced Alg. 4 MLP.

    Returns (y [B, D] fp64, K caches after Concat, V caches after Concat) so the
    result can be compared with ``ref.decode_layer`` and ``ref.gkvc_append``.
    """
    W = ref.widen_weights(weights)
    X = ref.bf16_bits_to_f64(x_bits)
    B, D = X.shape
    d = k_cache_bits.shape[-1]
    w_gu = interlace_gate_up(W["w_gate"], W["w_up"], tile)
    ys, kcs, vcs = [], [], []
    for b in range(B):
        p = int(pos[b])
        h = ref.rms_norm(X[b], W["attn_norm"], rms_eps)
        q = (W["w_q"] @ h).reshape(n_heads, d)
        k = (W["w_k"] @ h).reshape(n_kv_heads, d)
        v = (W["w_v"] @ h).reshape(n_kv_heads, d)
        o, kc, vc = attention_alg1(q, k, v, k_cache_bits[b], v_cache_bits[b], p, rope_base, n_kv_heads)
        h1 = X[b] + W["w_o"] @ o.reshape(-1)
        h2 = ref.rms_norm(h1, W["mlp_norm"], rms_eps)
        m, _ = mlp_interlaced(h2, w_gu, W["w_down"], tile)
        ys.append(h1 + m)
        kcs.append(kc)
        vcs.append(vc)
    return np.stack(ys), kcs, vcs
