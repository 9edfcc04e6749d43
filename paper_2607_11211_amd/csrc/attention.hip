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
//   * the K/V tile loads are issued right after the few prologue loads (the
//     cache does not depend on this step's projections);
//   * prologue: RoPE on the G query heads and on k, with shared cos/sin rows
//     in double precision (Alg. 3 joint RoPE; Eq. 22); the block that owns the
//     new position N_p rounds k and v to bf16 and writes them to slot N_p
//     (GKVC, Eq. 1). It uses the rounded values straight from LDS; slot N_p
//     is never read back from memory and no other block touches it;
//   * K/V tiles of 64 positions go global -> registers -> LDS with 16-byte
//     coalesced loads (a tile is one contiguous range of the [N_max, d] row
//     of (b, g)); a ring of up to three tiles is in flight in registers while
//     the current tile is computed from LDS;
//   * four lanes share a position (a quarter of d each): QK^T partials are
//     finished with two in-quad DPP moves, and each lane keeps an
//     online-softmax state (m, l, o-quarter) per query head;
//   * the block merges its lanes' states (DPP within each 16-lane row, then
//     the 16 rows through LDS) and writes (m, l, o) for its split.
// A second small kernel combines the splits of each (b, head) with the
// log-sum-exp identity. (Cross-block tickets are avoided on purpose: on this
// chip an agent-scope fence per block costs far more than a kernel boundary.)
#include "common.h"
#include "kernels.h"

#include <math.h>

namespace fasttps {

namespace {

constexpr int kThreads = 256;
constexpr int kTile = 64;         // positions per LDS tile
constexpr int kMaxSplits = 256;   // splits per (sequence, kv head); one combine thread each

constexpr int kRows = kThreads / 16;  // 16-lane DPP rows per block (4 positions each)

template <int D, int G>
struct alignas(16) AttnSmem {
  union {
    struct {
      uint16_t k[kTile][D + 8];  // padded rows: 16 extra bytes shift the banks
      uint16_t v[kTile][D + 8];
    } tile;
    float red[G][kRows][D];  // after the last tile: the rows' o sums
  };
  float q[G][D];
  uint16_t knew[D];
  uint16_t vnew[D];
  float rm[G][kRows];  // the rows' running max and sum
  float rl[G][kRows];
};

__device__ __forceinline__ float merge_factor(float m, float M) {
  return (m == -INFINITY) ? 0.f : __expf(m - M);
}

// Global -> registers: this thread's 16-byte chunks of the tile at t0.
// Only rows below P hold cached entries (commit keeps only those); the loads
// themselves are unconditional, with the row clamped into [t0, end), so the
// staging arrays stay in registers and every load stays in flight until its
// data is committed.
template <int D, int NPF>
__device__ __forceinline__ void tile_issue(v4u (&pk)[NPF], v4u (&pv)[NPF], const v4u* __restrict__ Kc,
                                           const v4u* __restrict__ Vc, int t0, int end, int tid) {
  constexpr int C8 = D / 8;
  const int last = min(kTile, end - t0) - 1;  // >= 0 since t0 < end
#pragma unroll
  for (int i = 0; i < NPF; ++i) {
    const int f = tid + kThreads * i;
    const int row = min(f / C8, last), c = f % C8;
    const size_t src = (size_t)(t0 + row) * C8 + c;
    pk[i] = Kc[src];
    pv[i] = Vc[src];
  }
}

// Registers -> LDS; the new entry (position P, if in this tile) comes from
// the rounded k/v already in LDS.
template <int D, int G, int NPF>
__device__ __forceinline__ void tile_commit(AttnSmem<D, G>& sm, const v4u (&pk)[NPF], const v4u (&pv)[NPF],
                                            int t0, int end, int P, int tid) {
  constexpr int C8 = D / 8;
  const int nvalid = min(kTile, end - t0);
  const int ncached = max(0, min(nvalid, P - t0));
#pragma unroll
  for (int i = 0; i < NPF; ++i) {
    const int f = tid + kThreads * i;
    const int row = f / C8, c = f % C8;
    if (row < ncached) {
      *reinterpret_cast<v4u*>(&sm.tile.k[row][c * 8]) = pk[i];
      *reinterpret_cast<v4u*>(&sm.tile.v[row][c * 8]) = pv[i];
    }
  }
  if (P >= t0 && P < t0 + nvalid && tid < 2 * C8) {
    const bool isv = tid >= C8;
    const int c = isv ? tid - C8 : tid;
    const v4u val = reinterpret_cast<const v4u*>(isv ? sm.vnew : sm.knew)[c];
    *reinterpret_cast<v4u*>(isv ? &sm.tile.v[P - t0][c * 8] : &sm.tile.k[P - t0][c * 8]) = val;
  }
}

// One tile: QK^T for the G query heads, online softmax, PV, for the
// position j = tid / 4 and the quarter seg = tid % 4 of d this lane owns.
template <int D, int G>
__device__ __forceinline__ void tile_compute(const AttnSmem<D, G>& sm, float (&m)[G], float (&l)[G],
                                             float (&o)[G][D / 4], int nvalid, int j, int seg, float scale) {
  constexpr int SEG = D / 4;
  const bool valid = j < nvalid;
  float sc[G];
#pragma unroll
  for (int h = 0; h < G; ++h) sc[h] = 0.f;
  if (valid) {
    const v4u* kr = reinterpret_cast<const v4u*>(&sm.tile.k[j][seg * SEG]);
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
  for (int h = 0; h < G; ++h) sc[h] = quad_sum(sc[h]) * scale;
  if (valid) {
    float vf[SEG];
    const v4u* vr = reinterpret_cast<const v4u*>(&sm.tile.v[j][seg * SEG]);
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
}

template <int D, int G, int NRING>
__global__ __launch_bounds__(kThreads) void attn_split_kernel(AttnArgs a) {
  constexpr int SEG = D / 4;                  // elements of a position row per lane
  constexpr int C8 = D / 8;                   // 16-byte chunks per row
  constexpr int HALF = D / 2;
  constexpr int NPF = kTile * C8 / kThreads;  // 16-byte chunks per thread per tile (K and V each)
  static_assert(SEG % 8 == 0, "a lane's quarter row must be whole 16-byte chunks");
  static_assert(NPF * kThreads == kTile * C8, "tile must split evenly over the block");
  __shared__ AttnSmem<D, G> sm;

  const int tid = threadIdx.x;
  const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int P = a.pos.p[b];
  const int ntot = P + 1;
  const int start = s * a.split_len;
  const int end = min(start + a.split_len, ntot);
  const int H = a.n_heads, Hkv = a.n_kv_heads;
  const size_t head_off = ((size_t)b * Hkv + g) * (size_t)a.max_seq * D;
  const v4u* Kc = reinterpret_cast<const v4u*>(a.k_cache + head_off);
  const v4u* Vc = reinterpret_cast<const v4u*>(a.v_cache + head_off);

  // ---- prologue operands first --------------------------------------------
  // Vector-memory loads retire in order: the few loads the prologue needs go
  // out before the tile stream, so waiting for them does not wait for tiles.
  const size_t rowlen = (size_t)(H + 2 * Hkv) * D;
  const float* qkv = a.qkv + (size_t)b * rowlen;
  const float* qg = qkv + (size_t)g * G * D;
  const float* kg = qkv + (size_t)H * D + (size_t)g * D;
  const float* vg = qkv + (size_t)(H + Hkv) * D + (size_t)g * D;
  const double* cs = a.rope_cos + (size_t)P * HALF;
  const double* sn = a.rope_sin + (size_t)P * HALF;
  const bool own_new = (start <= P) && (P < end);
  static_assert(G * HALF <= kThreads && D <= kThreads, "one prologue element per thread");
  const bool has_q = tid < G * HALF;
  const int pj = tid % HALF;
  double c_j = 0.0, s_j = 0.0;
  float q0 = 0.f, q1 = 0.f, k0 = 0.f, k1 = 0.f, v0 = 0.f;
  if (has_q) {
    c_j = cs[pj];
    s_j = sn[pj];
    q0 = qg[(tid / HALF) * D + pj];
    q1 = qg[(tid / HALF) * D + pj + HALF];
  }
  if (own_new) {
    if (tid < HALF) {
      k0 = kg[tid];
      k1 = kg[tid + HALF];
    }
    if (tid < D) v0 = vg[tid];
  }

  // ---- the first NRING tiles' loads ----------------------------------------
  // A ring of NRING tiles is in flight in registers; a tile's buffer is
  // refilled with the tile NRING ahead right after it is committed to LDS.
  v4u pk[NRING][NPF], pv[NRING][NPF];
#pragma unroll
  for (int k = 0; k < NRING; ++k)
    if (start + k * kTile < end) tile_issue<D, NPF>(pk[k], pv[k], Kc, Vc, start + k * kTile, end, tid);

  // ---- prologue: RoPE in double, rounding of the new K/V ------------------
  if (has_q) {
    const int hq = tid / HALF;
    sm.q[hq][pj] = (float)((double)q0 * c_j - (double)q1 * s_j);
    sm.q[hq][pj + HALF] = (float)((double)q1 * c_j + (double)q0 * s_j);
    if (own_new && tid < HALF) {
      sm.knew[pj] = f64_to_bf16((double)k0 * c_j - (double)k1 * s_j);
      sm.knew[pj + HALF] = f64_to_bf16((double)k1 * c_j + (double)k0 * s_j);
    }
  }
  if (own_new && tid < D) sm.vnew[tid] = f32_to_bf16(v0);
  __syncthreads();
  // GKVC append (Eq. 1): the one cache write of the step
  if (own_new && tid < 2 * C8) {
    const bool isv = tid >= C8;
    const int c = isv ? tid - C8 : tid;
    const v4u val = reinterpret_cast<const v4u*>(isv ? sm.vnew : sm.knew)[c];
    uint16_t* dst = (isv ? a.v_cache : a.k_cache) + head_off + (size_t)P * D;
    reinterpret_cast<v4u*>(dst)[c] = val;
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

  for (int t0 = start; t0 < end; t0 += NRING * kTile) {
#pragma unroll
    for (int k = 0; k < NRING; ++k) {
      const int tt = t0 + k * kTile;
      if (tt < end) {
        __syncthreads();  // every lane is done with the previous tile in LDS
        tile_commit<D, G, NPF>(sm, pk[k], pv[k], tt, end, P, tid);
        __syncthreads();
        if (tt + NRING * kTile < end) tile_issue<D, NPF>(pk[k], pv[k], Kc, Vc, tt + NRING * kTile, end, tid);
        tile_compute<D, G>(sm, m, l, o, min(kTile, end - tt), j, seg, a.scale);
      }
    }
  }

  // ---- merge: the 4 positions of each 16-lane row (DPP), then the rows ----
  static_assert(sizeof(float) * G * kRows * D <= sizeof(sm.tile), "merge space fits in the tile buffers");
  __syncthreads();  // every lane is done with the last tile: its LDS becomes merge space
  const int row = tid >> 4;
  const bool row_lead = (tid & 15) < 4;  // lane seg of position 0 of the row
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float Mr = row_stride4_max(m[h]);
    const float f = merge_factor(m[h], Mr);
    const float lr = row_stride4_sum(l[h] * f);
#pragma unroll
    for (int e = 0; e < SEG; ++e) o[h][e] = row_stride4_sum(o[h][e] * f);
    if (row_lead) {
      v4u* dst = reinterpret_cast<v4u*>(&sm.red[h][row][seg * SEG]);
#pragma unroll
      for (int c = 0; c < SEG / 4; ++c)
        dst[c] = v4u{__float_as_uint(o[h][4 * c]), __float_as_uint(o[h][4 * c + 1]), __float_as_uint(o[h][4 * c + 2]),
                     __float_as_uint(o[h][4 * c + 3])};
    }
    if ((tid & 15) == 0) {
      sm.rm[h][row] = Mr;
      sm.rl[h][row] = lr;
    }
  }
  __syncthreads();

  float* part_b = a.part + (size_t)b * H * a.nsplit_cap * (D + 2);
  for (int i = tid; i < G * D; i += kThreads) {
    const int h = i / D, e = i % D;
    float M = sm.rm[h][0];
#pragma unroll
    for (int r = 1; r < kRows; ++r) M = fmaxf(M, sm.rm[h][r]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      const float f = merge_factor(sm.rm[h][r], M);
      L = fmaf(sm.rl[h][r], f, L);
      O = fmaf(sm.red[h][r][e], f, O);
    }
    float* pr = part_b + ((size_t)(g * G + h) * a.nsplit_cap + s) * (D + 2);
    pr[2 + e] = O;
    if (e == 0) {
      pr[0] = M;
      pr[1] = L;
    }
  }
}

// o[b, h] = sum_s e^{m_s - M} o_s / sum_s e^{m_s - M} l_s,  M = max_s m_s.
// One block per (head, sequence). Every load is issued up front (the o rows
// do not depend on M), so the kernel costs one round trip: thread s reads
// split s's (m, l); thread (group, e) reads o_s[e] of the splits
// s = group, group + NG, ...
constexpr int kCombineThreads = 256;
constexpr int kCombineRegs = 16;  // splits per thread held in registers

template <int D>
__global__ __launch_bounds__(kCombineThreads) void attn_combine_kernel(const float* __restrict__ part, int nsplit,
                                                                       int nsplit_cap, int n_heads,
                                                                       float* __restrict__ o) {
  constexpr int NG = kCombineThreads / D;  // thread groups over the splits
  __shared__ float fac[kMaxSplits];
  __shared__ float red[kCombineThreads / kWave];
  __shared__ float osum[NG][D];
  const int tid = threadIdx.x;
  const int h = blockIdx.x, b = blockIdx.y;
  const float* ph = part + ((size_t)b * n_heads + h) * nsplit_cap * (D + 2);
  const int grp = tid / D, e = tid % D;
  float ov[kCombineRegs];
#pragma unroll
  for (int k = 0; k < kCombineRegs; ++k) {
    const int q = grp + NG * k;
    ov[k] = (grp < NG && q < nsplit) ? ph[(size_t)q * (D + 2) + 2 + e] : 0.f;
  }
  const float ms = tid < nsplit ? ph[(size_t)tid * (D + 2)] : -INFINITY;
  const float ls = tid < nsplit ? ph[(size_t)tid * (D + 2) + 1] : 0.f;
  float M = wave_max(ms);
  if ((tid & (kWave - 1)) == 0) red[tid / kWave] = M;
  __syncthreads();
  M = red[0];
#pragma unroll
  for (int w = 1; w < kCombineThreads / kWave; ++w) M = fmaxf(M, red[w]);
  const float f = merge_factor(ms, M);
  if (tid < nsplit) fac[tid] = f;
  const float L = block_sum(ls * f, red);  // its barriers also publish fac
  if (grp < NG) {
    float acc = 0.f;
#pragma unroll
    for (int k = 0; k < kCombineRegs; ++k) {
      const int q = grp + NG * k;
      if (q < nsplit) acc = fmaf(ov[k], fac[q], acc);
    }
    for (int q = grp + NG * kCombineRegs; q < nsplit; q += NG)
      acc = fmaf(ph[(size_t)q * (D + 2) + 2 + e], fac[q], acc);
    osum[grp][e] = acc;
  }
  __syncthreads();
  if (tid < D) {
    float O = 0.f;
#pragma unroll
    for (int g2 = 0; g2 < NG; ++g2) O += osum[g2][tid];
    o[((size_t)b * n_heads + h) * D + tid] = O / L;
  }
}

template <int D, int G>
hipError_t launch_dg(const AttnArgs& a, hipStream_t s, KernelEvents ev) {
  // tiles in flight per block: as many as the VGPR budget allows next to
  // the per-head softmax state (a tile is D / 2 VGPRs of K and V per lane)
  constexpr int NRING = (G == 1) ? 3 : (G == 2 ? 2 : 1);
  dim3 grid(a.nsplit, a.n_kv_heads, a.batch);
  return ext_launch(attn_split_kernel<D, G, NRING>, grid, dim3(kThreads), 0, s, ev, a);
}

template <int D>
hipError_t launch_d(const AttnArgs& a, hipStream_t s, KernelEvents ev) {
  switch (a.n_heads / a.n_kv_heads) {
    case 1: return launch_dg<D, 1>(a, s, ev);
    case 2: return launch_dg<D, 2>(a, s, ev);
    case 4: return launch_dg<D, 4>(a, s, ev);
    default: return hipErrorInvalidValue;
  }
}

template <int D>
hipError_t launch_combine_d(const AttnArgs& a, hipStream_t s, KernelEvents ev) {
  dim3 grid(a.n_heads, a.batch);
  return ext_launch(attn_combine_kernel<D>, grid, dim3(kCombineThreads), 0, s, ev, (const float*)a.part, a.nsplit,
                    a.nsplit_cap, a.n_heads, a.o);
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s, KernelEvents ev) {
  if (a.nsplit < 1 || a.nsplit > a.nsplit_cap || a.nsplit > kMaxSplits) return hipErrorInvalidValue;
  switch (a.head_dim) {
    case 64: return launch_d<64>(a, s, ev);
    case 96: return launch_d<96>(a, s, ev);
    case 128: return launch_d<128>(a, s, ev);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attention_combine(const AttnArgs& a, hipStream_t s, KernelEvents ev) {
  switch (a.head_dim) {
    case 64: return launch_combine_d<64>(a, s, ev);
    case 96: return launch_combine_d<96>(a, s, ev);
    case 128: return launch_combine_d<128>(a, s, ev);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fasttps
