// Fused SwiGLU MLP of the decode layer (gfx950).
//
// The paper's Fusion MLP (Section 3.2, Alg. 4) interlaces gate and up weights
// so that one larger projection yields, tile by tile, both halves that
// siLu_Mul combines (Eq. 29-31), and then runs the down projection (Eq. 32)
// over the stored intermediate. Here the intermediate never leaves the chip:
//   * block i owns the intermediate units [i*tk, i*tk + tk); its rows of the
//     interlaced W_gu are one contiguous [2 tk, D] slab (tk gate rows, then
//     the tk matching up rows), streamed with coalesced 16-byte loads;
//   * RMSNorm2 of h1 is computed by every block into LDS (fp32) while the
//     block's first weight loads are in flight;
//   * a = SiLU(gate) * up for the slab stays in LDS;
//   * the block then streams its tk rows of W_down^T ([K, D], so a K-slice
//     is contiguous) and writes a partial y over all D columns;
//   * a second small kernel adds the partials in a fixed order (so results
//     are bitwise reproducible) plus the residual h1, and rounds y to bf16.
#include "common.h"
#include "kernels.h"

#include <math.h>

namespace fasttps {

namespace {

constexpr int kThreads = 512;
constexpr int kGroup = 8;  // 16-byte chunks per lane per pass (4096 columns)
constexpr int kRpw = 2;    // gate/up rows per wave task

template <int BT>
__global__ __launch_bounds__(kThreads) void mlp_fused_kernel(MlpArgs a) {
  extern __shared__ float smem[];
  const int D = a.hidden;
  const int tk = a.tk;
  float* h2 = smem;                 // [BT][D]
  float* gu = h2 + BT * D;          // [BT][2 tk]
  float* red = gu + BT * 2 * tk;    // [16]
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int nwaves = blockDim.x / kWave;
  const int blk = blockIdx.x;
  const int k0 = blk * tk;
  const int tkb = min(tk, a.inter - k0);
  const int rows = 2 * tkb;
  const int b0 = blockIdx.y * BT;
  const int nb = min(BT, a.batch - b0);
  const int nch = D >> 3;
  const uint4* Wgu = reinterpret_cast<const uint4*>(a.w_gu) + (size_t)2 * k0 * nch;

  // 1. first gate/up loads of this wave (independent of h2)
  uint4 w[kRpw][kGroup];
  int r0 = wave * kRpw;
#pragma unroll
  for (int i = 0; i < kRpw; ++i)
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
      const int c = lane + kWave * j;
      w[i][j] = (r0 + i < rows && c < nch) ? Wgu[(size_t)(r0 + i) * nch + c] : make_uint4(0, 0, 0, 0);
    }

  // 2. RMSNorm2 prologue into LDS
  for (int b = 0; b < nb; ++b) {
    const float* hb = a.h1 + (size_t)(b0 + b) * D;
    float ss = 0.f;
    for (int c = threadIdx.x; c < D; c += blockDim.x) ss = fmaf(hb[c], hb[c], ss);
    const float tot = block_sum(ss, red);
    const float inv = 1.0f / sqrtf(tot / (float)D + a.eps);
    for (int c = threadIdx.x; c < D; c += blockDim.x) h2[b * D + c] = hb[c] * inv * bf16_to_f32(a.gamma[c]);
  }
  __syncthreads();

  // 3. gate/up rows: each wave takes kRpw rows at a time
  for (; r0 < rows; r0 += nwaves * kRpw) {
    float acc[kRpw][BT];
#pragma unroll
    for (int i = 0; i < kRpw; ++i)
#pragma unroll
      for (int b = 0; b < BT; ++b) acc[i][b] = 0.f;
    for (int base = 0; base < nch; base += kWave * kGroup) {
      if (base > 0) {
#pragma unroll
        for (int i = 0; i < kRpw; ++i)
#pragma unroll
          for (int j = 0; j < kGroup; ++j) {
            const int c = base + lane + kWave * j;
            w[i][j] = (r0 + i < rows && c < nch) ? Wgu[(size_t)(r0 + i) * nch + c] : make_uint4(0, 0, 0, 0);
          }
      }
#pragma unroll
      for (int j = 0; j < kGroup; ++j) {
        const int c = base + lane + kWave * j;
        if (c < nch) {
#pragma unroll
          for (int b = 0; b < BT; ++b) {
            if (b < nb) {
              const float4* hp = reinterpret_cast<const float4*>(h2 + b * D + 8 * c);
              const float4 x0 = hp[0], x1 = hp[1];
              const float h[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
              for (int i = 0; i < kRpw; ++i) acc[i][b] = fma8(w[i][j], h, acc[i][b]);
            }
          }
        }
      }
    }
#pragma unroll
    for (int i = 0; i < kRpw; ++i)
#pragma unroll
      for (int b = 0; b < BT; ++b) {
        const float v = wave_sum(acc[i][b]);
        if (lane == 0 && r0 + i < rows && b < nb) gu[b * 2 * tk + r0 + i] = v;
      }
    // loads for the next task of this wave
    const int rn = r0 + nwaves * kRpw;
    if (rn < rows) {
#pragma unroll
      for (int i = 0; i < kRpw; ++i)
#pragma unroll
        for (int j = 0; j < kGroup; ++j) {
          const int c = lane + kWave * j;
          w[i][j] = (rn + i < rows && c < nch) ? Wgu[(size_t)(rn + i) * nch + c] : make_uint4(0, 0, 0, 0);
        }
    }
  }
  __syncthreads();

  // 4. siLu_Mul on the slab: a = SiLU(gate) * up, kept in LDS (gate half is
  //    rows [0, tkb), up half rows [tkb, 2 tkb))
  float* act = gu;  // in place: a[b][t] overwrites gate[b][t]
  for (int i = threadIdx.x; i < nb * tkb; i += blockDim.x) {
    const int b = i / tkb, t = i % tkb;
    const float gt = gu[b * 2 * tk + t];
    const float up = gu[b * 2 * tk + tkb + t];
    const float av = gt / (1.0f + expf(-gt)) * up;
    act[b * 2 * tk + t] = av;
    if (a.a_dbg) a.a_dbg[(size_t)(b0 + b) * a.inter + k0 + t] = av;
  }
  __syncthreads();

  // 5. down projection of the slab: partial[blk][b][c] = sum_t W_down^T[k0+t][c] a[b][t]
  const uint4* Wd = reinterpret_cast<const uint4*>(a.w_downT) + (size_t)k0 * nch;
  for (int c = threadIdx.x; c < nch; c += blockDim.x) {
    float acc[BT][8];
#pragma unroll
    for (int b = 0; b < BT; ++b)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[b][e] = 0.f;
    int t = 0;
    for (; t + 8 <= tkb; t += 8) {
      uint4 wv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) wv[u] = Wd[(size_t)(t + u) * nch + c];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        float wf[8];
        unpack8(wv[u], wf);
#pragma unroll
        for (int b = 0; b < BT; ++b) {
          if (b < nb) {
            const float av = act[b * 2 * tk + t + u];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[b][e] = fmaf(wf[e], av, acc[b][e]);
          }
        }
      }
    }
    for (; t < tkb; ++t) {
      float wf[8];
      unpack8(Wd[(size_t)t * nch + c], wf);
#pragma unroll
      for (int b = 0; b < BT; ++b) {
        if (b < nb) {
          const float av = act[b * 2 * tk + t];
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[b][e] = fmaf(wf[e], av, acc[b][e]);
        }
      }
    }
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      if (b < nb) {
        float4* dst = reinterpret_cast<float4*>(a.partial + ((size_t)blk * a.batch + b0 + b) * D + 8 * c);
        dst[0] = make_float4(acc[b][0], acc[b][1], acc[b][2], acc[b][3]);
        dst[1] = make_float4(acc[b][4], acc[b][5], acc[b][6], acc[b][7]);
      }
    }
  }
}

template <int BT>
hipError_t launch_bt(const MlpArgs& a, hipStream_t s, KernelEvents ev) {
  dim3 grid(mlp_blocks(a.inter, a.tk), (a.batch + BT - 1) / BT);
  const size_t lds = ((size_t)BT * a.hidden + (size_t)BT * 2 * a.tk + 16) * sizeof(float);
  return ext_launch(mlp_fused_kernel<BT>, grid, dim3(kThreads), lds, s, ev, a);
}

// Partial sums: block = 64 slices x 4 column quads (16 columns); slice s adds
// partials s, s+64, ...; then a fixed tree over the 64 slices.
constexpr int kRedSlices = 64;

__global__ __launch_bounds__(256) void mlp_reduce_kernel(const float* __restrict__ h1,
                                                          const float* __restrict__ partial, int nblk,
                                                          int total, uint16_t* __restrict__ y) {
  __shared__ float4 buf[kRedSlices][4];
  const int quad = threadIdx.x & 3;
  const int slice = threadIdx.x >> 2;
  const int col4 = blockIdx.x * 4 + quad;  // index in float4 units over [batch * D]
  const int n4 = total >> 2;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  if (col4 < n4) {
    for (int p = slice; p < nblk; p += kRedSlices) {
      const float4 v = reinterpret_cast<const float4*>(partial + (size_t)p * total)[col4];
      acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
    }
  }
  buf[slice][quad] = acc;
  __syncthreads();
  for (int half = kRedSlices / 2; half >= 1; half >>= 1) {
    if (slice < half) {
      const float4 o = buf[slice + half][quad];
      float4 v = buf[slice][quad];
      v.x += o.x; v.y += o.y; v.z += o.z; v.w += o.w;
      buf[slice][quad] = v;
    }
    __syncthreads();
  }
  if (slice == 0 && col4 < n4) {
    const float4 r = reinterpret_cast<const float4*>(h1)[col4];
    const float4 v = buf[0][quad];
    const uint32_t lo = (uint32_t)f32_to_bf16(r.x + v.x) | ((uint32_t)f32_to_bf16(r.y + v.y) << 16);
    const uint32_t hi = (uint32_t)f32_to_bf16(r.z + v.z) | ((uint32_t)f32_to_bf16(r.w + v.w) << 16);
    reinterpret_cast<uint2*>(y)[col4] = make_uint2(lo, hi);
  }
}

}  // namespace

int mlp_blocks(int inter, int tk) { return (inter + tk - 1) / tk; }

hipError_t launch_mlp(const MlpArgs& a, hipStream_t s, KernelEvents ev) {
  // batch tile: h2 of BT sequences in LDS, at most 96 KB
  const size_t per = ((size_t)a.hidden + 2 * (size_t)a.tk) * sizeof(float);
  const int cap = (int)((96 * 1024) / per);
  const int want = a.batch < cap ? a.batch : cap;
  if (want >= 8) return launch_bt<8>(a, s, ev);
  if (want >= 4) return launch_bt<4>(a, s, ev);
  if (want >= 2) return launch_bt<2>(a, s, ev);
  return launch_bt<1>(a, s, ev);
}

hipError_t launch_mlp_reduce(const float* h1, const float* partial, int nblk, int batch, int hidden,
                             uint16_t* y, hipStream_t s, KernelEvents ev) {
  const int total = batch * hidden;  // multiple of 8
  const int n4 = total / 4;
  dim3 grid((n4 + 3) / 4);
  return ext_launch(mlp_reduce_kernel, grid, dim3(256), 0, s, ev, h1, partial, nblk, total, y);
}

}  // namespace fasttps
