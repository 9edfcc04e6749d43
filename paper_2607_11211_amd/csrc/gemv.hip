// Weight-streaming GEMV kernels of the decode layer (gfx950).
//
// At batch 1-8 the projections are matrix-vector products whose cost is the
// bf16 weight stream from HBM (Section 4.4 of the paper: token-phase MLP and
// projections are bound by weight movement). Layout of the work:
//   * a wavefront owns RPW consecutive rows; lane l reads the 16-byte chunks
//     l, l+64, ... of each row, so every load instruction of the wave covers
//     one contiguous kilobyte of a row (fully coalesced);
//   * all weight loads of a wave are issued before the block computes its
//     activation prologue (RMSNorm or fp32 copy into LDS), so the weight
//     stream does not wait for the prologue;
//   * products accumulate in fp32 against fp32 activations held in LDS, and
//     one cross-lane butterfly per row finishes the dot product.
#include "common.h"
#include "kernels.h"

namespace fasttps {

namespace {

constexpr int kThreads = 256;
constexpr int kGroup = 8;  // 16-byte chunks per lane per pass (4096 columns)

enum class Mode { kNormQkv, kResidual };

template <int BT, int RPW, Mode MODE>
__global__ __launch_bounds__(kThreads) void gemv_rows_kernel(GemvArgs a) {
  extern __shared__ float smem[];  // act [BT][din] fp32, then reduction scratch
  float* red = smem + BT * a.din;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int nwaves = blockDim.x / kWave;
  const int b0 = blockIdx.y * BT;
  const int nb = min(BT, a.batch - b0);
  const int r0 = (blockIdx.x * nwaves + wave) * RPW;
  const int nch = a.din >> 3;
  const uint4* W = reinterpret_cast<const uint4*>(a.w);

  // 1. first pass of weight loads, independent of the activation
  uint4 w[RPW][kGroup];
#pragma unroll
  for (int i = 0; i < RPW; ++i) {
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
      const int c = lane + kWave * j;
      w[i][j] = (r0 + i < a.rows && c < nch) ? W[(size_t)(r0 + i) * nch + c] : make_uint4(0, 0, 0, 0);
    }
  }

  // 2. activation prologue into LDS
  if (MODE == Mode::kNormQkv) {
    for (int b = 0; b < nb; ++b) {
      const uint16_t* xb = a.x_bf16 + (size_t)(b0 + b) * a.din;
      float ss = 0.f;
      for (int c = threadIdx.x; c < a.din; c += blockDim.x) {
        const float v = bf16_to_f32(xb[c]);
        ss = fmaf(v, v, ss);
      }
      const float tot = block_sum(ss, red);
      const float inv = 1.0f / sqrtf(tot / (float)a.din + a.eps);
      for (int c = threadIdx.x; c < a.din; c += blockDim.x)
        smem[b * a.din + c] = bf16_to_f32(xb[c]) * inv * bf16_to_f32(a.gamma[c]);
    }
  } else {
    for (int b = 0; b < nb; ++b) {
      const float4* src = reinterpret_cast<const float4*>(a.in_f32 + (size_t)(b0 + b) * a.din);
      float4* dst = reinterpret_cast<float4*>(smem + b * a.din);
      for (int c = threadIdx.x; c < (a.din >> 2); c += blockDim.x) dst[c] = src[c];
    }
  }
  __syncthreads();

  // 3. dot products, one pass of kGroup chunks per lane at a time
  float acc[RPW][BT];
#pragma unroll
  for (int i = 0; i < RPW; ++i)
#pragma unroll
    for (int b = 0; b < BT; ++b) acc[i][b] = 0.f;

  for (int base = 0; base < nch; base += kWave * kGroup) {
    if (base > 0) {
#pragma unroll
      for (int i = 0; i < RPW; ++i)
#pragma unroll
        for (int j = 0; j < kGroup; ++j) {
          const int c = base + lane + kWave * j;
          w[i][j] = (r0 + i < a.rows && c < nch) ? W[(size_t)(r0 + i) * nch + c] : make_uint4(0, 0, 0, 0);
        }
    }
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
      const int c = base + lane + kWave * j;
      if (c < nch) {
#pragma unroll
        for (int b = 0; b < BT; ++b) {
          if (b < nb) {
            const float4* hp = reinterpret_cast<const float4*>(smem + b * a.din + 8 * c);
            const float4 h0 = hp[0], h1 = hp[1];
            const float h[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
#pragma unroll
            for (int i = 0; i < RPW; ++i) acc[i][b] = fma8(w[i][j], h, acc[i][b]);
          }
        }
      }
    }
  }

  // 4. finish each row with a butterfly and store
#pragma unroll
  for (int i = 0; i < RPW; ++i) {
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      const float v = wave_sum(acc[i][b]);
      const int r = r0 + i;
      if (lane == 0 && b < nb && r < a.rows) {
        const size_t o = (size_t)(b0 + b) * a.rows + r;
        if (MODE == Mode::kNormQkv) {
          a.out[o] = v;
        } else {
          a.out[o] = bf16_to_f32(a.x_bf16[o]) + v;
        }
      }
    }
  }
}

template <Mode MODE, int BT>
hipError_t launch_bt(const GemvArgs& a, hipStream_t s, int rpw, KernelEvents ev) {
  const int nwaves = kThreads / kWave;
  const int rows_per_block = nwaves * rpw;
  dim3 grid((a.rows + rows_per_block - 1) / rows_per_block, (a.batch + BT - 1) / BT);
  const size_t lds = (size_t)BT * a.din * sizeof(float) + 64 * sizeof(float);
  if (rpw == 1) return ext_launch(gemv_rows_kernel<BT, 1, MODE>, grid, dim3(kThreads), lds, s, ev, a);
  return ext_launch(gemv_rows_kernel<BT, 2, MODE>, grid, dim3(kThreads), lds, s, ev, a);
}

template <Mode MODE>
hipError_t launch_mode(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  // batch tile: as many sequences as fit 64 KB of fp32 activations in LDS
  const int cap = (int)((65536 - 256) / ((size_t)a.din * sizeof(float)));
  const int want = a.batch < cap ? a.batch : cap;
  // two rows per wave when that still gives the chip >= 2 blocks per CU
  const int rpw = (a.rows / (4 * 2)) >= 512 ? 2 : 1;
  if (want >= 8) return launch_bt<MODE, 8>(a, s, rpw, ev);
  if (want >= 4) return launch_bt<MODE, 4>(a, s, rpw, ev);
  if (want >= 2) return launch_bt<MODE, 2>(a, s, rpw, ev);
  return launch_bt<MODE, 1>(a, s, rpw, ev);
}

}  // namespace

hipError_t launch_rmsnorm_qkv(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mode<Mode::kNormQkv>(a, s, ev);
}
hipError_t launch_oproj_residual(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mode<Mode::kResidual>(a, s, ev);
}

}  // namespace fasttps
