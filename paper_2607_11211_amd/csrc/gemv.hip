// Weight-streaming GEMV kernels of the decode layer (gfx950).
//
// At batch 1-8 the projections are matrix-vector products whose cost is the
// bf16 weight stream from HBM (Section 4.4 of the paper: token-phase MLP and
// projections are bound by weight movement). Layout of the work:
//   * one block per CU-share of rows: block b owns rows [b R / n, (b+1) R / n);
//     within it the rows are dealt to the waves round-robin, to waves 1..15
//     only when they can hold them all;
//   * lane l reads the 16-byte chunks l, l+64, ... of a row, so every load
//     instruction of a wave covers one contiguous kilobyte (fully coalesced);
//   * each wave keeps a ring of NBUF rows in flight in registers (up to the
//     VGPR budget): a row's buffer is refilled with the wave's next row as
//     soon as its products are taken, before the cross-lane reduction;
//   * the activation prologue (RMSNorm of x, or the fp32 attention output) is
//     built in LDS by wave 0 alone, before it issues weight loads, while the
//     other waves already stream weights. Vector-memory loads retire in
//     order, so a prologue load queued behind the weight loads would wait for
//     all of them; this keeps the weight stream independent of the prologue;
//   * products accumulate in fp32 against the fp32 activation in LDS, and one
//     cross-lane butterfly per row finishes each dot product.
#include "common.h"
#include "kernels.h"

namespace fasttps {

namespace {

enum class Mode { kNormQkv, kResidual };

constexpr int kNumCu = 256;

template <int MAXCH>
__device__ __forceinline__ void load_row(v4u (&w)[MAXCH], const v4u* __restrict__ W, int r, int re, int nch,
                                         int lane) {
#pragma unroll
  for (int j = 0; j < MAXCH; ++j) {
    const int c = lane + kWave * j;
    w[j] = (r < re && c < nch) ? W[(size_t)r * nch + c] : v4u{0u, 0u, 0u, 0u};
  }
}

template <int BT, int MAXCH>
__device__ __forceinline__ void dot_row(float (&acc)[BT], const v4u (&w)[MAXCH], const float* act, int din, int nb,
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
          const float4* hp = reinterpret_cast<const float4*>(act + b * din + 8 * c);
          const float4 h0 = hp[0], h1 = hp[1];
          float s = acc[b];
          s = fmaf(wf[0], h0.x, s);
          s = fmaf(wf[1], h0.y, s);
          s = fmaf(wf[2], h0.z, s);
          s = fmaf(wf[3], h0.w, s);
          s = fmaf(wf[4], h1.x, s);
          s = fmaf(wf[5], h1.y, s);
          s = fmaf(wf[6], h1.z, s);
          s = fmaf(wf[7], h1.w, s);
          acc[b] = s;
        }
      }
    }
  }
}

template <int BT, Mode MODE>
__device__ __forceinline__ void store_row(const float (&acc)[BT], const GemvArgs& a, int r, int b0, int nb, int lane) {
#pragma unroll
  for (int b = 0; b < BT; ++b) {
    const float v = wave_sum(acc[b]);
    if (lane == 0 && b < nb) {
      const size_t o = (size_t)(b0 + b) * a.rows + r;
      if (MODE == Mode::kNormQkv)
        a.out[o] = v;
      else
        a.out[o] = bf16_to_f32(a.x_bf16[o]) + v;
    }
  }
}

// Wave 0: activation of the batch tile into LDS as fp32 [BT][din].
template <int BT, int MAXCH, Mode MODE>
__device__ __forceinline__ void prologue_wave0(float* act, const GemvArgs& a, int b0, int nb, int lane) {
  const int nch = a.din >> 3;
  if (MODE == Mode::kNormQkv) {
    // h = x / sqrt(mean(x^2) + eps) * gamma   (RMSNorm1)
    // x rows and gamma go out in one batch of loads (one round trip when
    // din <= 512 MAXCH); then sum of squares, scale, store to LDS
    const v4u* gv = reinterpret_cast<const v4u*>(a.gamma);
    for (int b = 0; b < nb; ++b) {
      const v4u* xv = reinterpret_cast<const v4u*>(a.x_bf16 + (size_t)(b0 + b) * a.din);
      float ss = 0.f;
      for (int base = 0; base < nch; base += kWave * MAXCH) {
        v4u xs[MAXCH];
#pragma unroll
        for (int j = 0; j < MAXCH; ++j) {
          const int c = base + lane + kWave * j;
          xs[j] = c < nch ? xv[c] : v4u{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int j = 0; j < MAXCH; ++j) {
          const int c = base + lane + kWave * j;
          float f[8];
          unpack8(xs[j], f);
#pragma unroll
          for (int e = 0; e < 8; ++e) ss = fmaf(f[e], f[e], ss);
          if (c < nch) {
            float4* d = reinterpret_cast<float4*>(act + b * a.din + 8 * c);
            d[0] = make_float4(f[0], f[1], f[2], f[3]);
            d[1] = make_float4(f[4], f[5], f[6], f[7]);
          }
        }
      }
      ss = wave_sum(ss);
      const float inv = 1.0f / sqrtf(ss / (float)a.din + a.eps);
      for (int base = 0; base < nch; base += kWave * MAXCH) {
        v4u gs[MAXCH];
#pragma unroll
        for (int j = 0; j < MAXCH; ++j) {
          const int c = base + lane + kWave * j;
          gs[j] = c < nch ? gv[c] : v4u{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int j = 0; j < MAXCH; ++j) {
          const int c = base + lane + kWave * j;
          if (c < nch) {
            float g[8];
            unpack8(gs[j], g);
            float4* d = reinterpret_cast<float4*>(act + b * a.din + 8 * c);
            float4 v0 = d[0], v1 = d[1];
            v0 = make_float4(v0.x * inv * g[0], v0.y * inv * g[1], v0.z * inv * g[2], v0.w * inv * g[3]);
            v1 = make_float4(v1.x * inv * g[4], v1.y * inv * g[5], v1.z * inv * g[6], v1.w * inv * g[7]);
            d[0] = v0;
            d[1] = v1;
          }
        }
      }
    }
  } else {
    // fp32 copy of the attention output
    for (int b = 0; b < nb; ++b) {
      const float4* src = reinterpret_cast<const float4*>(a.in_f32 + (size_t)(b0 + b) * a.din);
      float4* dst = reinterpret_cast<float4*>(act + b * a.din);
      const int n4 = a.din >> 2;
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
          if (c < n4) dst[c] = t[j];
        }
      }
    }
  }
}

template <int BT, int MAXCH, int NW, int NBUF, Mode MODE>
__global__ __launch_bounds__(NW * kWave) void gemv_kernel(GemvArgs a) {
  extern __shared__ float act[];  // [BT][din] fp32
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int b0 = blockIdx.y * BT;
  const int nb = min(BT, a.batch - b0);
  const int nch = a.din >> 3;
  const int rb = (int)((long)blockIdx.x * a.rows / gridDim.x);
  const int re = (int)((long)(blockIdx.x + 1) * a.rows / gridDim.x);
  const v4u* W = reinterpret_cast<const v4u*>(a.w);
  // Rows go to waves 1..NW-1 when they can hold the block's share in their
  // NBUF row buffers, so wave 0 (the prologue wave) has no weight stream.
  const int nworkers = (re - rb <= NBUF * (NW - 1)) ? NW - 1 : NW;
  const int widx = (nworkers == NW) ? NW - 1 - wave : wave - 1;  // -1: no rows
  const int r0 = rb + widx;
  const int step = nworkers;

  v4u w[NBUF][MAXCH];
  if (wave == 0) prologue_wave0<BT, MAXCH, MODE>(act, a, b0, nb, lane);
  if (widx >= 0) {
#pragma unroll
    for (int k = 0; k < NBUF; ++k) load_row<MAXCH>(w[k], W, r0 + k * step, re, nch, lane);
  }
  __syncthreads();
  if (widx < 0) return;

  for (int i0 = 0; r0 + i0 * step < re; i0 += NBUF) {
#pragma unroll
    for (int k = 0; k < NBUF; ++k) {
      const int r = r0 + (i0 + k) * step;
      if (r < re) {
        float acc[BT];
        dot_row<BT, MAXCH>(acc, w[k], act, a.din, nb, nch, lane);
        load_row<MAXCH>(w[k], W, r + NBUF * step, re, nch, lane);
        store_row<BT, MODE>(acc, a, r, b0, nb, lane);
      }
    }
  }
}

template <int BT, int MAXCH, Mode MODE>
hipError_t launch_bt(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  // Each wave holds NBUF rows in flight, as many as its VGPR budget allows
  // (a row is 4 MAXCH VGPRs; 128 VGPRs per lane with 16 waves, 256 with 8).
  constexpr int NW = MAXCH <= 8 ? 16 : 8;
  constexpr int NBUF = MAXCH <= 2 ? 4 : (MAXCH <= 6 ? 3 : 2);
  const int nblk = a.rows < kNumCu ? a.rows : kNumCu;
  dim3 grid(nblk, (a.batch + BT - 1) / BT);
  const size_t lds = (size_t)BT * a.din * sizeof(float);
  return ext_launch(gemv_kernel<BT, MAXCH, NW, NBUF, MODE>, grid, dim3(NW * kWave), lds, s, ev, a);
}

template <int MAXCH, Mode MODE>
hipError_t launch_ch(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  // batch tile: as many sequences as fit 64 KB of fp32 activations in LDS
  const int cap = (int)(65536 / ((size_t)a.din * sizeof(float)));
  const int want = a.batch < cap ? a.batch : cap;
  if constexpr (MAXCH <= 4) {  // 8 sequences fit the LDS tile only when din <= 2048
    if (want >= 8) return launch_bt<8, MAXCH, MODE>(a, s, ev);
  }
  if constexpr (MAXCH <= 8) {  // 4 sequences fit the LDS tile only when din <= 4096
    if (want >= 4) return launch_bt<4, MAXCH, MODE>(a, s, ev);
  }
  if (want >= 2) return launch_bt<2, MAXCH, MODE>(a, s, ev);
  return launch_bt<1, MAXCH, MODE>(a, s, ev);
}

template <Mode MODE>
hipError_t launch_mode(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  const int chunks_per_lane = (a.din / 8 + kWave - 1) / kWave;
  if (chunks_per_lane <= 1) return launch_ch<1, MODE>(a, s, ev);
  if (chunks_per_lane <= 2) return launch_ch<2, MODE>(a, s, ev);
  if (chunks_per_lane <= 4) return launch_ch<4, MODE>(a, s, ev);
  if (chunks_per_lane <= 6) return launch_ch<6, MODE>(a, s, ev);
  if (chunks_per_lane <= 8) return launch_ch<8, MODE>(a, s, ev);
  if (chunks_per_lane <= 16) return launch_ch<16, MODE>(a, s, ev);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_rmsnorm_qkv(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mode<Mode::kNormQkv>(a, s, ev);
}
hipError_t launch_oproj_residual(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mode<Mode::kResidual>(a, s, ev);
}

}  // namespace fasttps
