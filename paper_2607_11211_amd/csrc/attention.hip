// Decode attention with joint RoPE, in-place cache append and split-KV (gfx950).
//
// The paper's TPSFLAT (Alg. 3, Section 3.1.2) runs RoPE, the K append, QK^T,
// softmax and PV for one head inside one core's L1. One head's work is far
// too small for a 256-CU chip, so here the softmax-independent axis the paper
// uses (heads) is combined with a split of the cached positions:
//   grid = (split, kv head g, sequence b); a block covers positions
//   [s*L, s*L + L) of one (b, g) for all G = H/H_kv query heads of that KV
//   head, so each K/V byte is read from HBM once (grouped-query attention).
// Per block:
//   * prologue: RoPE on the G query heads and on k, with shared cos/sin rows
//     in double precision (Alg. 3 joint RoPE; Eq. 22); the block that owns the
//     new position N_p rounds k and v to bf16 and writes them to slot N_p
//     (GKVC, Eq. 1). It uses the rounded values straight from LDS; slot N_p
//     is never read back from memory and no other block touches it;
//   * K/V tiles of 64 positions are copied to LDS with 16-byte coalesced loads
//     (each tile is one contiguous range of the [N_max, d] row of (b, g));
//   * four lanes share a position (a quarter of d each): QK^T partials are
//     finished with two butterflies, and each lane keeps an online-softmax
//     state (m, l, o-quarter) per query head;
//   * the block merges its lanes' states, writes (m, l, o) for its split, and
//     the last split of (b, g) to finish (atomic ticket) combines the splits
//     with the log-sum-exp identity and writes o. It resets its ticket.
#include "common.h"
#include "kernels.h"

#include <math.h>

namespace fasttps {

namespace {

constexpr int kThreads = 256;
constexpr int kTile = 64;        // positions per LDS tile
constexpr int kMaxSplits = 256;  // bound on splits per (b, g)

template <int D, int G>
struct alignas(16) AttnSmem {
  uint16_t kt[kTile][D + 8];   // padded rows: 16 extra bytes shift the banks
  uint16_t vt[kTile][D + 8];
  float q[G][D];
  uint16_t knew[D];
  uint16_t vnew[D];
  float wm[4][G];
  float wl[4][G];
  float wo[4][G][D];
  float fac[G][kMaxSplits];
  float lsum[G];
  int last;
};

__device__ __forceinline__ float merge_factor(float m, float M) {
  return (m == -INFINITY) ? 0.f : __expf(m - M);
}

template <int D, int G>
__global__ __launch_bounds__(kThreads) void attn_split_kernel(AttnArgs a) {
  constexpr int SEG = D / 4;     // elements of a position row per lane
  constexpr int C8 = D / 8;      // 16-byte chunks per row
  constexpr int HALF = D / 2;
  __shared__ AttnSmem<D, G> sm;

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int P = a.pos.p[b];
  const int ntot = P + 1;
  const int start = s * a.split_len;
  const int end = min(start + a.split_len, ntot);
  const int H = a.n_heads, Hkv = a.n_kv_heads;
  const size_t rowlen = (size_t)(H + 2 * Hkv) * D;
  const float* qkv = a.qkv + (size_t)b * rowlen;
  const float* qg = qkv + (size_t)g * G * D;
  const float* kg = qkv + (size_t)H * D + (size_t)g * D;
  const float* vg = qkv + (size_t)(H + Hkv) * D + (size_t)g * D;
  const double* cs = a.rope_cos + (size_t)P * HALF;
  const double* sn = a.rope_sin + (size_t)P * HALF;
  const size_t head_off = ((size_t)b * Hkv + g) * (size_t)a.max_seq * D;
  const bool own_new = (start <= P) && (P < end);

  // ---- prologue: RoPE (double), append of the new K/V --------------------
  for (int i = tid; i < G * HALF; i += kThreads) {
    const int hq = i / HALF, j = i % HALF;
    const double c = cs[j], sv = sn[j];
    const double x0 = qg[hq * D + j], x1 = qg[hq * D + j + HALF];
    sm.q[hq][j] = (float)(x0 * c - x1 * sv);
    sm.q[hq][j + HALF] = (float)(x1 * c + x0 * sv);
  }
  if (own_new) {
    for (int j = tid; j < HALF; j += kThreads) {
      const double c = cs[j], sv = sn[j];
      const double k0 = kg[j], k1 = kg[j + HALF];
      sm.knew[j] = f64_to_bf16(k0 * c - k1 * sv);
      sm.knew[j + HALF] = f64_to_bf16(k1 * c + k0 * sv);
    }
    for (int j = tid; j < D; j += kThreads) sm.vnew[j] = f32_to_bf16(vg[j]);
  }
  __syncthreads();
  if (own_new && tid < 2 * C8) {
    const bool isv = tid >= C8;
    const int c = isv ? tid - C8 : tid;
    const uint4 val = reinterpret_cast<const uint4*>(isv ? sm.vnew : sm.knew)[c];
    uint16_t* dst = (isv ? a.v_cache : a.k_cache) + head_off + (size_t)P * D;
    reinterpret_cast<uint4*>(dst)[c] = val;
  }

  // ---- main loop over tiles ------------------------------------------------
  const int j = tid >> 2, seg = tid & 3;
  float m[G], l[G], o[G][SEG];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY;
    l[h] = 0.f;
#pragma unroll
    for (int e = 0; e < SEG; ++e) o[h][e] = 0.f;
  }
  const uint4* Kc = reinterpret_cast<const uint4*>(a.k_cache + head_off);
  const uint4* Vc = reinterpret_cast<const uint4*>(a.v_cache + head_off);

  for (int t0 = start; t0 < end; t0 += kTile) {
    const int nvalid = min(kTile, end - t0);
    const int ncached = max(0, min(nvalid, P - t0));
    for (int f = tid; f < ncached * C8; f += kThreads) {
      const int row = f / C8, c = f % C8;
      const size_t src = (size_t)(t0 + row) * C8 + c;
      *reinterpret_cast<uint4*>(&sm.kt[row][c * 8]) = Kc[src];
      *reinterpret_cast<uint4*>(&sm.vt[row][c * 8]) = Vc[src];
    }
    if (P >= t0 && P < t0 + nvalid && tid < 2 * C8) {
      const bool isv = tid >= C8;
      const int c = isv ? tid - C8 : tid;
      const uint4 val = reinterpret_cast<const uint4*>(isv ? sm.vnew : sm.knew)[c];
      *reinterpret_cast<uint4*>(isv ? &sm.vt[P - t0][c * 8] : &sm.kt[P - t0][c * 8]) = val;
    }
    __syncthreads();

    const bool valid = j < nvalid;
    float sc[G];
#pragma unroll
    for (int h = 0; h < G; ++h) sc[h] = 0.f;
    if (valid) {
      const uint4* kr = reinterpret_cast<const uint4*>(&sm.kt[j][seg * SEG]);
#pragma unroll
      for (int c = 0; c < SEG / 8; ++c) {
        float kf[8];
        unpack8(kr[c], kf);
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float* qh = &sm.q[h][seg * SEG + c * 8];
#pragma unroll
          for (int e = 0; e < 8; ++e) sc[h] = fmaf(qh[e], kf[e], sc[h]);
        }
      }
    }
#pragma unroll
    for (int h = 0; h < G; ++h) {
      sc[h] += __shfl_xor(sc[h], 1, kWave);
      sc[h] += __shfl_xor(sc[h], 2, kWave);
      sc[h] *= a.scale;
    }
    if (valid) {
      float vf[SEG];
      const uint4* vr = reinterpret_cast<const uint4*>(&sm.vt[j][seg * SEG]);
#pragma unroll
      for (int c = 0; c < SEG / 8; ++c) unpack8(vr[c], vf + 8 * c);
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float mn = fmaxf(m[h], sc[h]);
        const float cf = merge_factor(m[h], mn);
        const float p = __expf(sc[h] - mn);
        l[h] = fmaf(l[h], cf, p);
#pragma unroll
        for (int e = 0; e < SEG; ++e) o[h][e] = fmaf(o[h][e], cf, p * vf[e]);
        m[h] = mn;
      }
    }
    __syncthreads();
  }

  // ---- merge the 16 position groups of each wave, then the 4 waves --------
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float M = m[h];
    M = fmaxf(M, __shfl_xor(M, 4, kWave));
    M = fmaxf(M, __shfl_xor(M, 8, kWave));
    M = fmaxf(M, __shfl_xor(M, 16, kWave));
    M = fmaxf(M, __shfl_xor(M, 32, kWave));
    const float f = merge_factor(m[h], M);
    float lv = l[h] * f;
#pragma unroll
    for (int msk = 4; msk < kWave; msk <<= 1) lv += __shfl_xor(lv, msk, kWave);
#pragma unroll
    for (int e = 0; e < SEG; ++e) {
      float ov = o[h][e] * f;
#pragma unroll
      for (int msk = 4; msk < kWave; msk <<= 1) ov += __shfl_xor(ov, msk, kWave);
      if (lane < 4) sm.wo[wave][h][lane * SEG + e] = ov;
    }
    if (lane == 0) {
      sm.wm[wave][h] = M;
      sm.wl[wave][h] = lv;
    }
  }
  __syncthreads();

  const int nsplit = a.nsplit;
  float* part_b = a.part + (size_t)b * H * a.nsplit_cap * (D + 2);
  for (int i = tid; i < G * D; i += kThreads) {
    const int h = i / D, e = i % D;
    float M = sm.wm[0][h];
    for (int w = 1; w < 4; ++w) M = fmaxf(M, sm.wm[w][h]);
    float L = 0.f, O = 0.f;
    for (int w = 0; w < 4; ++w) {
      const float f = merge_factor(sm.wm[w][h], M);
      L = fmaf(sm.wl[w][h], f, L);
      O = fmaf(sm.wo[w][h][e], f, O);
    }
    float* pr = part_b + ((size_t)(g * G + h) * a.nsplit_cap + s) * (D + 2);
    pr[2 + e] = O;
    if (e == 0) {
      pr[0] = M;
      pr[1] = L;
    }
  }

  // ---- last split of (b, g) combines --------------------------------------
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    const unsigned prev = atomicAdd(&a.tickets[b * Hkv + g], 1u);
    sm.last = (prev == (unsigned)(nsplit - 1));
  }
  __syncthreads();
  if (!sm.last) return;
  __threadfence();

  if (tid < G) {
    const int h = tid;
    const float* ph = part_b + (size_t)(g * G + h) * a.nsplit_cap * (D + 2);
    float M = -INFINITY;
    for (int q = 0; q < nsplit; ++q) M = fmaxf(M, __builtin_nontemporal_load(ph + (size_t)q * (D + 2)));
    float L = 0.f;
    for (int q = 0; q < nsplit; ++q) {
      const float f = merge_factor(__builtin_nontemporal_load(ph + (size_t)q * (D + 2)), M);
      sm.fac[h][q] = f;
      L = fmaf(__builtin_nontemporal_load(ph + (size_t)q * (D + 2) + 1), f, L);
    }
    sm.lsum[h] = L;
  }
  __syncthreads();
  for (int i = tid; i < G * D; i += kThreads) {
    const int h = i / D, e = i % D;
    const float* ph = part_b + (size_t)(g * G + h) * a.nsplit_cap * (D + 2);
    float O = 0.f;
    for (int q = 0; q < nsplit; ++q) O = fmaf(__builtin_nontemporal_load(ph + (size_t)q * (D + 2) + 2 + e), sm.fac[h][q], O);
    a.o[(size_t)b * H * D + (size_t)(g * G + h) * D + e] = O / sm.lsum[h];
  }
  if (tid == 0) a.tickets[b * Hkv + g] = 0u;
}

template <int D, int G>
hipError_t launch_dg(const AttnArgs& a, hipStream_t s) {
  dim3 grid(a.nsplit, a.n_kv_heads, a.batch);
  hipLaunchKernelGGL((attn_split_kernel<D, G>), grid, dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_d(const AttnArgs& a, hipStream_t s) {
  switch (a.n_heads / a.n_kv_heads) {
    case 1: return launch_dg<D, 1>(a, s);
    case 2: return launch_dg<D, 2>(a, s);
    case 4: return launch_dg<D, 4>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.nsplit < 1 || a.nsplit > kMaxSplits || a.nsplit > a.nsplit_cap) return hipErrorInvalidValue;
  switch (a.head_dim) {
    case 64: return launch_d<64>(a, s);
    case 96: return launch_d<96>(a, s);
    case 128: return launch_d<128>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fasttps
