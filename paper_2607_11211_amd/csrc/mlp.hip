// Fusion MLP of the decode layer, gate/up part (gfx950).
//
// The paper's Fusion MLP (Section 3.2, Alg. 4) interlaces gate and up weights
// so that one larger projection yields, tile by tile, both halves that
// siLu_Mul combines (Eq. 29-31); the result h^sm (here `a`, fp32) is stored,
// and the down projection (Eq. 32) reads it back as a separate step. Here:
//   * block i owns the intermediate units [i*tk, i*tk + tk); its rows of the
//     interlaced W_gu are one contiguous [2 tk, D] slab (tk gate rows, then
//     the tk matching up rows), streamed with coalesced 16-byte loads;
//   * RMSNorm2 of h1 is computed into LDS (fp32) by wave 0 of every block
//     while the other waves already stream the slab (vector-memory loads
//     retire in order, so the prologue's loads go out before any weight load
//     of wave 0);
//   * the gate and up sums of the slab meet in LDS; siLu_Mul writes a.
// The down projection with the residual and the bf16 rounding of y is the
// GEMV kernel's down mode: a full-row GEMV over W_down in its own [D, K]
// layout, so no partial sums cross blocks.
#include "common.h"
#include "kernels.h"

#include <math.h>

namespace fasttps {

namespace {

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
__global__ __launch_bounds__(NW * kWave) void mlp_gate_up_kernel(MlpArgs a) {
  extern __shared__ __attribute__((aligned(16))) float smem[];
  const int D = a.hidden;
  const int tk = a.tk;
  float* h2 = smem;         // [BT][D]
  float* gu = h2 + BT * D;  // [BT][2 tk]
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

  // 2. gate/up slab: rows dealt round-robin to the waves (to waves 1..NW-1
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

  __syncthreads();  // gate and up sums of the slab complete

  // siLu_Mul on the slab (gate half rows [0, tkb), up half rows [tkb, 2 tkb))
  for (int i = tid; i < nb * tkb; i += blockDim.x) {
    const int b = i / tkb, t = i % tkb;
    const float gt = gu[b * 2 * tk + t];
    const float up = gu[b * 2 * tk + tkb + t];
    a.a[(size_t)(b0 + b) * a.inter + k0 + t] = gt / (1.0f + expf(-gt)) * up;
  }
}

template <int BT, int MAXCH>
hipError_t launch_bt(const MlpArgs& a, hipStream_t s, KernelEvents ev) {
  constexpr int NW = 16;
  // row buffers per wave within the 128-VGPR budget (a row is 4 MAXCH VGPRs)
  constexpr int NBUF = MAXCH <= 2 ? 4 : (MAXCH <= 6 ? (BT >= 4 ? 2 : 3) : (MAXCH <= 8 ? 2 : 1));
  dim3 grid(mlp_blocks(a.inter, a.tk), (a.batch + BT - 1) / BT);
  const size_t lds = ((size_t)BT * a.hidden + (size_t)BT * 2 * a.tk) * sizeof(float);
  return ext_launch(mlp_gate_up_kernel<BT, MAXCH, NW, NBUF>, grid, dim3(NW * kWave), lds, s, ev, a);
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

}  // namespace

int mlp_blocks(int inter, int tk) { return (inter + tk - 1) / tk; }

hipError_t launch_mlp_gate_up(const MlpArgs& a, hipStream_t s, KernelEvents ev) {
  const int chunks_per_lane = (a.hidden / 8 + kWave - 1) / kWave;
  if (chunks_per_lane <= 1) return launch_ch<1>(a, s, ev);
  if (chunks_per_lane <= 2) return launch_ch<2>(a, s, ev);
  if (chunks_per_lane <= 4) return launch_ch<4>(a, s, ev);
  if (chunks_per_lane <= 6) return launch_ch<6>(a, s, ev);
  if (chunks_per_lane <= 8) return launch_ch<8>(a, s, ev);
  if (chunks_per_lane <= 16) return launch_ch<16>(a, s, ev);
  return hipErrorInvalidValue;
}

}  // namespace fasttps
