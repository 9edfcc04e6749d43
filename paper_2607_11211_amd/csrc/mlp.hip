// Fused SwiGLU MLP of the decode layer (gfx950).
//
// The paper's Fusion MLP (Section 3.2, Alg. 4) interlaces gate and up weights
// so that one larger projection yields, tile by tile, both halves that
// siLu_Mul combines (Eq. 29-31), and then runs the down projection (Eq. 32)
// over the stored intermediate. Here the intermediate never leaves the chip:
//   * block i owns the intermediate units [i*tk, i*tk + tk); its rows of the
//     interlaced W_gu are one contiguous [2 tk, D] slab (tk gate rows, then
//     the tk matching up rows), streamed with coalesced 16-byte loads;
//   * RMSNorm2 of h1 is computed into LDS (fp32) by wave 0 of every block
//     while the other waves already stream the slab (vector-memory loads
//     retire in order, so the prologue's loads go out before any weight load
//     of wave 0);
//   * a = SiLU(gate) * up for the slab stays in LDS;
//   * the block then streams its tk rows of W_down^T ([K, D], so a K-slice
//     is contiguous; the first rows are already in flight before the
//     SiLU barrier) and writes a partial y over all D columns;
//   * a second small kernel adds the partials in a fixed order (so results
//     are bitwise reproducible) plus the residual h1, and rounds y to bf16.
#include "common.h"
#include "kernels.h"

#include <math.h>

#include <algorithm>

namespace fasttps {

namespace {

constexpr int kDownPf = 16;  // W_down^T rows in flight per thread in the down phase

template <int MAXCH>
__device__ __forceinline__ void load_row(v4u (&w)[MAXCH], const v4u* __restrict__ W, int r, int rows, int nch,
                                         int lane) {
#pragma unroll
  for (int j = 0; j < MAXCH; ++j) {
    const int c = lane + kWave * j;
    w[j] = (r < rows && c < nch) ? W[(size_t)r * nch + c] : v4u{0u, 0u, 0u, 0u};
  }
}

// gate/up row against h2 (LDS): per-lane partial dot products
template <int BT, int MAXCH>
__device__ __forceinline__ void gu_dot(float (&acc)[BT], const v4u (&w)[MAXCH], const float* h2, int D, int nb,
                                       int nch, int lane) {
#pragma unroll
  for (int b = 0; b < BT; ++b) acc[b] = 0.f;
#pragma unroll
  for (int j = 0; j < MAXCH; ++j) {
    const int c = lane + kWave * j;
    if (c < nch) {
      float wf[8];
      unpack8(w[j], wf);
#pragma unroll
      for (int b = 0; b < BT; ++b) {
        if (b < nb) {
          const float4* hp = reinterpret_cast<const float4*>(h2 + b * D + 8 * c);
          const float4 x0 = hp[0], x1 = hp[1];
          float s = acc[b];
          s = fmaf(wf[0], x0.x, s);
          s = fmaf(wf[1], x0.y, s);
          s = fmaf(wf[2], x0.z, s);
          s = fmaf(wf[3], x0.w, s);
          s = fmaf(wf[4], x1.x, s);
          s = fmaf(wf[5], x1.y, s);
          s = fmaf(wf[6], x1.z, s);
          s = fmaf(wf[7], x1.w, s);
          acc[b] = s;
        }
      }
    }
  }
}

// finish a gate/up row with a butterfly over the wave and store it to gu
template <int BT>
__device__ __forceinline__ void gu_store(const float (&acc)[BT], float* gu, int r, int tk, int nb, int lane) {
#pragma unroll
  for (int b = 0; b < BT; ++b) {
    const float v = wave_sum(acc[b]);
    if (lane == 0 && b < nb) gu[b * 2 * tk + r] = v;
  }
}

template <int BT, int MAXCH, int NW, int NBUF>
__global__ __launch_bounds__(NW * kWave) void mlp_fused_kernel(MlpArgs a) {
  extern __shared__ __attribute__((aligned(16))) float smem[];
  const int D = a.hidden;
  const int tk = a.tk;
  float* h2 = smem;         // [BT][D]; reused for the second down-phase partial
  float* gu = h2 + BT * D;  // [BT][2 tk]
  // the first NL rows of this block's W_down^T slab, copied verbatim
  uint16_t* dsl = reinterpret_cast<uint16_t*>(gu + BT * 2 * tk);
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int blk = blockIdx.x;
  const int k0 = blk * tk;
  const int tkb = min(tk, a.inter - k0);
  const int rows = 2 * tkb;
  const int b0 = blockIdx.y * BT;
  const int nb = min(BT, a.batch - b0);
  const int nch = D >> 3;
  const v4u* Wgu = reinterpret_cast<const v4u*>(a.w_gu) + (size_t)2 * k0 * nch;
  const v4u* Wd = reinterpret_cast<const v4u*>(a.w_downT) + (size_t)k0 * nch;

  // 1. wave 0: RMSNorm2 of h1 into LDS, before it issues weight loads
  if (wave == 0) {
    const v4u* gv = reinterpret_cast<const v4u*>(a.gamma);
    for (int b = 0; b < nb; ++b) {
      const float4* src = reinterpret_cast<const float4*>(a.h1 + (size_t)(b0 + b) * D);
      float4* dst = reinterpret_cast<float4*>(h2 + b * D);
      const int n4 = D >> 2;
      float ss = 0.f;
      for (int base = 0; base < n4; base += kWave * 16) {
        float4 t[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int c = base + lane + kWave * j;
          t[j] = c < n4 ? src[c] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int c = base + lane + kWave * j;
          ss = fmaf(t[j].x, t[j].x, fmaf(t[j].y, t[j].y, fmaf(t[j].z, t[j].z, fmaf(t[j].w, t[j].w, ss))));
          if (c < n4) dst[c] = t[j];
        }
      }
      ss = wave_sum(ss);
      const float inv = 1.0f / sqrtf(ss / (float)D + a.eps);
      for (int base = 0; base < nch; base += kWave * 8) {
        v4u gs[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int c = base + lane + kWave * j;
          gs[j] = c < nch ? gv[c] : v4u{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int c = base + lane + kWave * j;
          if (c < nch) {
            float g[8];
            unpack8(gs[j], g);
            float4* d = reinterpret_cast<float4*>(h2 + b * D + 8 * c);
            float4 v0 = d[0], v1 = d[1];
            v0 = make_float4(v0.x * inv * g[0], v0.y * inv * g[1], v0.z * inv * g[2], v0.w * inv * g[3]);
            v1 = make_float4(v1.x * inv * g[4], v1.y * inv * g[5], v1.z * inv * g[6], v1.w * inv * g[7]);
            d[0] = v0;
            d[1] = v1;
          }
        }
      }
    }
  }

  // 2. the first NL rows of the W_down^T slab go straight to LDS
  //    (global_load_lds: no registers held); they are needed only after the
  //    gate/up phase, so they stream alongside it. One wave instruction moves
  //    one contiguous KiB; lane i lands at base + 16 i.
  const int NL = min(a.lds_rows, tkb);
  {
    const int nv = NL * nch;                 // 16-byte chunks to copy
    const int nq = (nv + kWave - 1) / kWave; // wave instructions
    for (int q = wave; q < nq; q += NW) {
      const int idx = q * kWave + lane;
      if (idx < nv)
        __builtin_amdgcn_global_load_lds(
            static_cast<const void*>(Wd + idx),
            (__attribute__((address_space(3))) void*)(dsl + (size_t)q * kWave * 8),
            16, 0, 0);
    }
  }

  // 3. gate/up slab: rows dealt round-robin to the waves (to waves 1..NW-1
  //    only when their NBUF row buffers can hold the whole slab); each wave
  //    keeps a ring of NBUF rows in flight, refilled as rows are consumed.
  {
    const int nworkers = (rows <= NBUF * (NW - 1)) ? NW - 1 : NW;
    const int widx = (nworkers == NW) ? NW - 1 - wave : wave - 1;  // -1: no rows
    const int r0 = widx;
    const int step = nworkers;
    v4u w[NBUF][MAXCH];
    if (widx >= 0) {
#pragma unroll
      for (int k = 0; k < NBUF; ++k) load_row<MAXCH>(w[k], Wgu, r0 + k * step, rows, nch, lane);
    }
    __syncthreads();  // h2 ready
    if (widx >= 0) {
      for (int i0 = 0; r0 + i0 * step < rows; i0 += NBUF) {
#pragma unroll
        for (int k = 0; k < NBUF; ++k) {
          const int r = r0 + (i0 + k) * step;
          if (r < rows) {
            float acc[BT];
            gu_dot<BT, MAXCH>(acc, w[k], h2, D, nb, nch, lane);
            load_row<MAXCH>(w[k], Wgu, r + NBUF * step, rows, nch, lane);
            gu_store<BT>(acc, gu, r, tk, nb, lane);
          }
        }
      }
    }
  }

  // 4. down phase layout: thread (group g, 16-byte column chunk c); group g
  //    owns LDS rows [g NL / NG, (g+1) NL / NG) and register rows
  //    NL + [g NR / NG, (g+1) NR / NG), NR = tkb - NL. The first register
  //    rows go out before the barrier: they do not depend on the activation.
  const int NG = min(2, (int)blockDim.x / nch);
  const int grp = tid / nch, c = tid % nch;
  const bool active = grp < NG;
  const int NR = tkb - NL;
  const int l0 = active ? grp * NL / NG : 0;
  const int l1 = active ? (grp + 1) * NL / NG : 0;
  const int t0 = active ? NL + grp * NR / NG : 0;
  const int t1 = active ? NL + (grp + 1) * NR / NG : 0;
  v4u wd[kDownPf];
#pragma unroll
  for (int u = 0; u < kDownPf; ++u)
    wd[u] = (t0 + u < t1) ? Wd[(size_t)(t0 + u) * nch + c] : v4u{0u, 0u, 0u, 0u};
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's LDS copies have landed
  __syncthreads();  // gu complete; the LDS slab rows of every wave visible

  // 5. siLu_Mul on the slab (gate half rows [0, tkb), up half rows [tkb, 2 tkb)),
  //    in place over the gate half
  for (int i = tid; i < nb * tkb; i += blockDim.x) {
    const int b = i / tkb, t = i % tkb;
    const float gt = gu[b * 2 * tk + t];
    const float up = gu[b * 2 * tk + tkb + t];
    const float av = gt / (1.0f + expf(-gt)) * up;
    gu[b * 2 * tk + t] = av;
    if (a.a_dbg) a.a_dbg[(size_t)(b0 + b) * a.inter + k0 + t] = av;
  }
  __syncthreads();  // a complete; h2 no longer needed

  // 6. partial y over all D columns: sum_t W_down^T[k0 + t][c] a[t]
  float acc[BT][8];
#pragma unroll
  for (int b = 0; b < BT; ++b)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[b][e] = 0.f;
  for (int t = l0; t < l1; ++t) {
    float wf[8];
    unpack8(*reinterpret_cast<const v4u*>(dsl + (size_t)t * D + 8 * c), wf);
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      if (b < nb) {
        const float av = gu[b * 2 * tk + t];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[b][e] = fmaf(wf[e], av, acc[b][e]);
      }
    }
  }
  for (int t = t0; t < t1; t += kDownPf) {
#pragma unroll
    for (int u = 0; u < kDownPf; ++u) {
      if (t + u < t1) {
        float wf[8];
        unpack8(wd[u], wf);
#pragma unroll
        for (int b = 0; b < BT; ++b) {
          if (b < nb) {
            const float av = gu[b * 2 * tk + t + u];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[b][e] = fmaf(wf[e], av, acc[b][e]);
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kDownPf; ++u) {
      const int tn = t + kDownPf + u;
      wd[u] = (tn < t1) ? Wd[(size_t)tn * nch + c] : v4u{0u, 0u, 0u, 0u};
    }
  }
  // group 1 hands its partial to group 0 through LDS (the h2 area)
  if (active && grp == 1) {
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      if (b < nb) {
        float4* d = reinterpret_cast<float4*>(h2 + b * D + 8 * c);
        d[0] = make_float4(acc[b][0], acc[b][1], acc[b][2], acc[b][3]);
        d[1] = make_float4(acc[b][4], acc[b][5], acc[b][6], acc[b][7]);
      }
    }
  }
  __syncthreads();
  if (active && grp == 0) {
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      if (b < nb) {
        if (NG > 1) {
          const float4* p = reinterpret_cast<const float4*>(h2 + b * D + 8 * c);
          const float4 p0 = p[0], p1 = p[1];
          acc[b][0] += p0.x; acc[b][1] += p0.y; acc[b][2] += p0.z; acc[b][3] += p0.w;
          acc[b][4] += p1.x; acc[b][5] += p1.y; acc[b][6] += p1.z; acc[b][7] += p1.w;
        }
        float4* dst = reinterpret_cast<float4*>(a.partial + ((size_t)blk * a.batch + b0 + b) * D + 8 * c);
        dst[0] = make_float4(acc[b][0], acc[b][1], acc[b][2], acc[b][3]);
        dst[1] = make_float4(acc[b][4], acc[b][5], acc[b][6], acc[b][7]);
      }
    }
  }
}

constexpr size_t kLdsBudget = 160 * 1024;  // LDS of one CU on gfx950

template <int BT, int MAXCH>
hipError_t launch_bt(const MlpArgs& a, hipStream_t s, KernelEvents ev) {
  constexpr int NW = 16;
  // row buffers per wave within the 128-VGPR budget (a row is 4 MAXCH VGPRs)
  constexpr int NBUF = MAXCH <= 2 ? 4 : (MAXCH <= 6 ? (BT >= 4 ? 2 : 3) : (MAXCH <= 8 ? 2 : 1));
  dim3 grid(mlp_blocks(a.inter, a.tk), (a.batch + BT - 1) / BT);
  const size_t fixed = ((size_t)BT * a.hidden + (size_t)BT * 2 * a.tk) * sizeof(float);
  const size_t row = (size_t)a.hidden * sizeof(uint16_t);
  MlpArgs b = a;
  b.lds_rows = fixed < kLdsBudget ? (int)std::min<size_t>((size_t)a.tk, (kLdsBudget - fixed) / row) : 0;
  const size_t lds = fixed + (size_t)b.lds_rows * row;
  return ext_launch(mlp_fused_kernel<BT, MAXCH, NW, NBUF>, grid, dim3(NW * kWave), lds, s, ev, b);
}

template <int MAXCH>
hipError_t launch_ch(const MlpArgs& a, hipStream_t s, KernelEvents ev) {
  // batch tile: h2 of BT sequences in LDS, at most 96 KB
  const size_t per = ((size_t)a.hidden + 2 * (size_t)a.tk) * sizeof(float);
  const int cap = (int)((96 * 1024) / per);
  const int want = a.batch < cap ? a.batch : cap;
  if constexpr (MAXCH <= 8) {  // wider rows take one sequence per tile (VGPR and LDS budget)
    if (want >= 4) return launch_bt<4, MAXCH>(a, s, ev);
    if (want >= 2) return launch_bt<2, MAXCH>(a, s, ev);
  }
  return launch_bt<1, MAXCH>(a, s, ev);
}

// Partial sums: one wave per 4-column quad; lane s adds partials s, s+64,
// ... (all loads issued together), then a fixed butterfly over the 64 lanes,
// so the result does not depend on timing.
constexpr int kRedLoads = 8;  // partials per lane held in registers

__global__ __launch_bounds__(256) void mlp_reduce_kernel(const float* __restrict__ h1,
                                                          const float* __restrict__ partial, int nblk,
                                                          int total, uint16_t* __restrict__ y) {
  const int lane = threadIdx.x & (kWave - 1);
  const int col4 = blockIdx.x * 4 + threadIdx.x / kWave;  // float4 index over [batch * D]
  const int n4 = total >> 2;
  if (col4 >= n4) return;  // whole wave exits together
  const float4* P = reinterpret_cast<const float4*>(partial);
  float4 v[kRedLoads];
#pragma unroll
  for (int k = 0; k < kRedLoads; ++k) {
    const int p = lane + kWave * k;
    v[k] = p < nblk ? P[(size_t)p * n4 + col4] : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float4 acc = v[0];
#pragma unroll
  for (int k = 1; k < kRedLoads; ++k) {
    acc.x += v[k].x; acc.y += v[k].y; acc.z += v[k].z; acc.w += v[k].w;
  }
  for (int p = lane + kWave * kRedLoads; p < nblk; p += kWave) {
    const float4 t = P[(size_t)p * n4 + col4];
    acc.x += t.x; acc.y += t.y; acc.z += t.z; acc.w += t.w;
  }
  acc.x = wave_sum(acc.x);
  acc.y = wave_sum(acc.y);
  acc.z = wave_sum(acc.z);
  acc.w = wave_sum(acc.w);
  if (lane == 0) {
    const float4 r = reinterpret_cast<const float4*>(h1)[col4];
    const uint32_t lo = (uint32_t)f32_to_bf16(r.x + acc.x) | ((uint32_t)f32_to_bf16(r.y + acc.y) << 16);
    const uint32_t hi = (uint32_t)f32_to_bf16(r.z + acc.z) | ((uint32_t)f32_to_bf16(r.w + acc.w) << 16);
    reinterpret_cast<uint2*>(y)[col4] = make_uint2(lo, hi);
  }
}

}  // namespace

int mlp_blocks(int inter, int tk) { return (inter + tk - 1) / tk; }

hipError_t launch_mlp(const MlpArgs& a, hipStream_t s, KernelEvents ev) {
  const int chunks_per_lane = (a.hidden / 8 + kWave - 1) / kWave;
  if (chunks_per_lane <= 1) return launch_ch<1>(a, s, ev);
  if (chunks_per_lane <= 2) return launch_ch<2>(a, s, ev);
  if (chunks_per_lane <= 4) return launch_ch<4>(a, s, ev);
  if (chunks_per_lane <= 6) return launch_ch<6>(a, s, ev);
  if (chunks_per_lane <= 8) return launch_ch<8>(a, s, ev);
  if (chunks_per_lane <= 16) return launch_ch<16>(a, s, ev);
  return hipErrorInvalidValue;
}

hipError_t launch_mlp_reduce(const float* h1, const float* partial, int nblk, int batch, int hidden,
                             uint16_t* y, hipStream_t s, KernelEvents ev) {
  const int total = batch * hidden;  // multiple of 8
  const int n4 = total / 4;
  dim3 grid((n4 + 3) / 4);
  return ext_launch(mlp_reduce_kernel, grid, dim3(256), 0, s, ev, h1, partial, nblk, total, y);
}

}  // namespace fasttps
