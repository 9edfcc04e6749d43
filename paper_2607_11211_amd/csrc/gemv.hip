// Weight-streaming GEMV kernels of the decode layer (gfx950).
//
// At batch 1-8 the projections are matrix-vector products whose cost is the
// bf16 weight stream from HBM (Section 4.4 of the paper: token-phase MLP and
// projections are bound by weight movement). Layout of the work:
//   * rows are dealt to the blocks round-robin (block b takes rows b, b + G,
//     b + 2G, ... of a grid of G blocks), so at any moment the chip reads a
//     compact window of the matrix; within a block the rows go round-robin to
//     waves 1..NW-1;
//   * lane l reads the 16-byte chunks l, l+64, ... of a row, so every load
//     instruction of a wave covers one contiguous kilobyte (fully coalesced);
//   * each wave keeps a ring of NBUF rows in flight in registers (up to the
//     VGPR budget): a row's buffer is refilled with the wave's next row as
//     soon as its products are taken, before the cross-lane reduction;
//   * a row longer than 64 MAXCH chunks (the down projection's K) is taken
//     in segments of 64 MAXCH chunks; the ring then holds (row, segment)
//     items in the wave's order and the sum of a row is carried across its
//     segments;
//   * the activation (RMSNorm of x, or a copy of an fp32 vector) is built in
//     LDS from slices that every wave loads before its first weight load: a
//     wave's loads return in the order they were issued, so a prologue load
//     queued behind the weight stream would wait for most of it;
//   * every global load in the kernel is issued unconditionally (clamped or
//     dead addresses where there is nothing to load), so the number of loads
//     in flight is known on every path and the compiler waits for exactly the
//     loads a step needs rather than for all of them;
//   * products accumulate in fp32 against the fp32 activation in LDS, and one
//     cross-lane reduction per row finishes each dot product.
#include "common.h"
#include "kernels.h"

namespace fasttps {

namespace {

// kNormQkv:     out = W RMSNorm(x)            (fp32)
// kResidual:    out = x + W act               (x bf16, act fp32; fp32 out)
// kDownResidual: y = bf16(res + W act)       (res, act fp32; bf16 out)
enum class Mode { kNormQkv, kResidual, kDownResidual };

constexpr int kNumCu = 256;

// The 16-byte chunks cbase + lane + 64 j of row r. Every lane issues every
// load, so the number of loads in flight is the same on every path and the
// compiler's wait before each ring slot counts exactly the loads issued after
// that slot's: chunks past the row are clamped to its last chunk (the dot
// product skips them), and a dead slot (live false) points every lane at the
// first 16 bytes of one of the block's rows (`rdead`), one cache line per
// instruction, different for every wave.
template <int MAXCH>
__device__ __forceinline__ void load_row(v4u (&w)[MAXCH], const v4u* __restrict__ W, bool live, int r, int rdead,
                                         int nch, int cbase, int lane) {
  const v4u* row = W + (size_t)(live ? r : rdead) * nch;
  const int cmax = live ? nch - 1 : 0;
#pragma unroll
  for (int j = 0; j < MAXCH; ++j) w[j] = row[min(cbase + lane + kWave * j, cmax)];
}

// acc[b] += the lane's share of row . act[b] over chunks cbase + lane + 64 j
template <int BT, int MAXCH>
__device__ __forceinline__ void dot_row(float (&acc)[BT], const v4u (&w)[MAXCH], const float* act, int din, int nb,
                                        int nch, int cbase, int lane) {
#pragma unroll
  for (int j = 0; j < MAXCH; ++j) {
    const int c = cbase + lane + kWave * j;
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

// Finish a row: the cross-lane sum of each sequence's partial products goes
// to the block's result buffer in LDS (global stores wait until the ring is
// drained, which keeps every global access of the loop a load).
template <int BT>
__device__ __forceinline__ void finish_row(const float (&acc)[BT], float* res, int nres, int idx, int nb, int lane) {
#pragma unroll
  for (int b = 0; b < BT; ++b) {
    const float v = wave_sum(acc[b]);
    if (lane == 0 && b < nb) res[b * nres + idx] = v;
  }
}

// The block's rows blk + G i of every sequence of the tile, from LDS to the
// output (with the residual and the rounding the mode asks for).
template <int BT, Mode MODE>
__device__ __forceinline__ void write_rows(const float* res, const float* resid, int nres, const GemvArgs& a,
                                           int blk, int G, int nrow, int b0, int nb) {
  for (int t = threadIdx.x; t < nb * nrow; t += blockDim.x) {
    const int b = t / nrow, i = t % nrow;
    const float v = res[b * nres + i];
    const size_t o = (size_t)(b0 + b) * a.rows + blk + (size_t)G * i;
    if (MODE == Mode::kNormQkv)
      a.out[o] = v;
    else if (MODE == Mode::kResidual)
      a.out[o] = resid[b * nres + i] + v;
    else
      a.out_bf16[o] = f32_to_bf16(resid[b * nres + i] + v);
  }
}

// The prologue's source, as n 16-byte chunks: the x rows of the tile and the
// gain (norm mode, bf16, copied to the stage), or the fp32 activation rows
// (copied to act). Chunk q of the x rows and gain: row q / nch, chunk q % nch.
template <int BT, Mode MODE>
__device__ __forceinline__ const v4u* prologue_chunk(const GemvArgs& a, int b0, int nb, int q) {
  const int nch = a.din >> 3;
  if (MODE == Mode::kNormQkv) {
    const int r = q / nch, c = q % nch;
    return r < nb ? reinterpret_cast<const v4u*>(a.x_bf16 + (size_t)(b0 + r) * a.din) + c
                  : reinterpret_cast<const v4u*>(a.gamma) + c;
  }
  return reinterpret_cast<const v4u*>(a.in_f32 + (size_t)b0 * a.din) + q;
}

// Wave `wave` takes chunks [wave CP 64, (wave + 1) CP 64) of the n: lane l
// loads chunks base + l + 64 j, j < CP (clamped to the last chunk).
template <int BT, int CP, Mode MODE>
__device__ __forceinline__ void slice_load(v4u (&t)[CP], const GemvArgs& a, int b0, int nb, int n, int wave,
                                           int lane) {
#pragma unroll
  for (int j = 0; j < CP; ++j) t[j] = *prologue_chunk<BT, MODE>(a, b0, nb, min((wave * CP + j) * kWave + lane, n - 1));
}

// The slice into LDS: the stage in norm mode (x rows, then the gain at row
// BT), act otherwise.
template <int BT, int CP, Mode MODE>
__device__ __forceinline__ void slice_store(const v4u (&t)[CP], float* act, uint16_t* stage, const GemvArgs& a,
                                            int nb, int n, int wave, int lane) {
  const int nch = a.din >> 3;
#pragma unroll
  for (int j = 0; j < CP; ++j) {
    const int q = (wave * CP + j) * kWave + lane;
    if (q < n) {
      if (MODE == Mode::kNormQkv) {
        const int r = q / nch, c = q % nch;
        reinterpret_cast<v4u*>(stage + (size_t)(r < nb ? r : BT) * a.din)[c] = t[j];
      } else {
        reinterpret_cast<v4u*>(act)[q] = t[j];
      }
    }
  }
}

// Norm mode, wave 0, from the stage: h = x / sqrt(mean(x^2) + eps) * gamma
// (RMSNorm1) into act as fp32.
template <int BT>
__device__ __forceinline__ void rmsnorm_from_stage(float* act, const uint16_t* stage, const GemvArgs& a, int nb,
                                                   int lane) {
  const int nch = a.din >> 3;
  const v4u* gv = reinterpret_cast<const v4u*>(stage + (size_t)BT * a.din);
  for (int b = 0; b < nb; ++b) {
    const v4u* xv = reinterpret_cast<const v4u*>(stage + (size_t)b * a.din);
    float ss = 0.f;
    for (int c = lane; c < nch; c += kWave) {
      float f[8];
      unpack8(xv[c], f);
#pragma unroll
      for (int e = 0; e < 8; ++e) ss = fmaf(f[e], f[e], ss);
    }
    ss = wave_sum(ss);
    const float inv = 1.0f / sqrtf(ss / (float)a.din + a.eps);
    for (int c = lane; c < nch; c += kWave) {
      float f[8], g[8];
      unpack8(xv[c], f);
      unpack8(gv[c], g);
      float4* d = reinterpret_cast<float4*>(act + b * a.din + 8 * c);
      d[0] = make_float4(f[0] * inv * g[0], f[1] * inv * g[1], f[2] * inv * g[2], f[3] * inv * g[3]);
      d[1] = make_float4(f[4] * inv * g[4], f[5] * inv * g[5], f[6] * inv * g[6], f[7] * inv * g[7]);
    }
  }
}

template <int BT, int MAXCH, int NW, int NBUF, int CP, Mode MODE>
__global__ __launch_bounds__(NW * kWave) void gemv_kernel(GemvArgs a) {
  // LDS: act [BT][din] fp32 | stage [(BT + 1)][din] bf16 (norm mode) | res [BT][nres] fp32
  //      | resid [BT][nres] fp32 (residual modes)
  extern __shared__ __attribute__((aligned(16))) float act[];
  uint16_t* stage = reinterpret_cast<uint16_t*>(act + (size_t)BT * a.din);
  const int G = gridDim.x, blk = blockIdx.x;
  const int nres = (a.rows + G - 1) / G;
  float* res = act + (size_t)BT * a.din + (MODE == Mode::kNormQkv ? (size_t)(BT + 1) * a.din / 2 : 0);
  float* resid = res + (size_t)BT * nres;  // residual modes: [BT][nres]
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int b0 = blockIdx.y * BT;
  const int nb = min(BT, a.batch - b0);
  const int nch = a.din >> 3;
  constexpr int kSeg = kWave * MAXCH;  // chunks per row segment
  const int nseg = (nch + kSeg - 1) / kSeg;
  const int nrow = a.rows > blk ? (a.rows - 1 - blk) / G + 1 : 0;  // rows blk + G i, i < nrow
  const v4u* W = reinterpret_cast<const v4u*>(a.w);
  // wave w >= 1 takes the block's rows i = w - 1, w - 1 + (NW - 1), ..., each
  // in nseg segments: item t is row i = w - 1 + (NW - 1) (t / nseg), segment t % nseg
  constexpr int kWorkers = NW - 1;
  const int widx = wave - 1;
  const int nitems = (widx >= 0 && widx < nrow) ? ((nrow - 1 - widx) / kWorkers + 1) * nseg : 0;
  // the row a dead load points at: one of the block's own rows (nrow >= 1,
  // since the grid has at most `rows` blocks), a different one per wave
  const int rdead = blk + G * (max(widx, 0) % nrow);

  // prologue slices first, then the weight ring, then the slices into LDS
  const int ncopy = MODE == Mode::kNormQkv ? (nb + 1) * nch : nb * a.din / 4;
  v4u t[CP];
  slice_load<BT, CP, MODE>(t, a, b0, nb, ncopy, wave, lane);
  __builtin_amdgcn_sched_barrier(0);  // keep the slice loads ahead of the weight loads

  // (block-local row, segment) of the item in each ring slot
  int sidx[NBUF], sseg[NBUF];
  v4u w[NBUF][MAXCH];
  // every wave issues the prefill (dead loads where it has no items), so the
  // slice stores below wait for the slice loads only
#pragma unroll
  for (int k = 0; k < NBUF; ++k) {
    sidx[k] = widx + kWorkers * (k / nseg);
    sseg[k] = k % nseg;
    load_row<MAXCH>(w[k], W, k < nitems, blk + G * sidx[k], rdead, nch, sseg[k] * kSeg, lane);
  }
  slice_store<BT, CP, MODE>(t, act, stage, a, nb, ncopy, wave, lane);
  __syncthreads();
  if (MODE == Mode::kNormQkv) {
    if (wave == 0) rmsnorm_from_stage<BT>(act, stage, a, nb, lane);
    __syncthreads();  // activation ready
  }

  // wave 0 (no rows of its own) fetches the residual of the block's rows
  // into LDS while the others stream weights
  if (MODE != Mode::kNormQkv && wave == 0) {
    for (int t = lane; t < nb * nrow; t += kWave) {
      const int b = t / nrow, i = t % nrow;
      const size_t o = (size_t)(b0 + b) * a.rows + blk + (size_t)G * i;
      resid[b * nres + i] = MODE == Mode::kResidual ? bf16_to_f32(a.x_bf16[o]) : a.res_f32[o];
    }
  }

  if (nitems > 0) {
    float acc[BT];
#pragma unroll
    for (int b = 0; b < BT; ++b) acc[b] = 0.f;
    for (int i0 = 0; i0 < nitems; i0 += NBUF) {
#pragma unroll
      for (int k = 0; k < NBUF; ++k) {
        const bool live = i0 + k < nitems;
        const int idx = sidx[k], seg = sseg[k];
        if (live) dot_row<BT, MAXCH>(acc, w[k], act, a.din, nb, nch, seg * kSeg, lane);
        // refill the slot with the item NBUF further on (a dead load past the end)
        int ni = idx, ns = seg + NBUF;
        while (ns >= nseg) {
          ns -= nseg;
          ni += kWorkers;
        }
        sidx[k] = ni;
        sseg[k] = ns;
        load_row<MAXCH>(w[k], W, i0 + k + NBUF < nitems, blk + G * ni, rdead, nch, ns * kSeg, lane);
        if (live && seg == nseg - 1) {
          finish_row<BT>(acc, res, nres, idx, nb, lane);
#pragma unroll
          for (int b = 0; b < BT; ++b) acc[b] = 0.f;
        }
      }
    }
  }
  __syncthreads();  // every row of the block (and its residual) is in LDS
  write_rows<BT, MODE>(res, resid, nres, a, blk, G, nrow, b0, nb);
}

// prologue chunks per lane: the smallest of 1, 2, 4, 8 that covers the
// prologue's 16-byte chunks over NW waves (at most 8 KB per wave)
template <int BT, int MAXCH, int NW, int NBUF, Mode MODE>
hipError_t launch_cp(const GemvArgs& a, dim3 grid, size_t lds, hipStream_t s, KernelEvents ev) {
  const int nb = a.batch < BT ? a.batch : BT;
  const long n = MODE == Mode::kNormQkv ? (long)(nb + 1) * (a.din / 8) : (long)nb * a.din / 4;
  const long per = (n + (long)NW * kWave - 1) / ((long)NW * kWave);
  if (per <= 1) return ext_launch(gemv_kernel<BT, MAXCH, NW, NBUF, 1, MODE>, grid, dim3(NW * kWave), lds, s, ev, a);
  if (per <= 2) return ext_launch(gemv_kernel<BT, MAXCH, NW, NBUF, 2, MODE>, grid, dim3(NW * kWave), lds, s, ev, a);
  if (per <= 4) return ext_launch(gemv_kernel<BT, MAXCH, NW, NBUF, 4, MODE>, grid, dim3(NW * kWave), lds, s, ev, a);
  if (per <= 8) return ext_launch(gemv_kernel<BT, MAXCH, NW, NBUF, 8, MODE>, grid, dim3(NW * kWave), lds, s, ev, a);
  return hipErrorInvalidValue;
}

template <int BT, int MAXCH, Mode MODE>
hipError_t launch_bt(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  // 16 waves; each keeps about 8 KB of weights in flight (NBUF items of
  // MAXCH KB): more outstanding loads per CU only queue up in the memory
  // system and make the stream slower.
  constexpr int NW = 16;
  constexpr int NBUF = MAXCH >= 6 ? 1 : (MAXCH >= 4 ? 2 : (MAXCH >= 2 ? 4 : 8));
  const int nblk = a.rows < kNumCu ? a.rows : kNumCu;
  dim3 grid(nblk, (a.batch + BT - 1) / BT);
  size_t lds = (size_t)BT * a.din * sizeof(float);
  if (MODE == Mode::kNormQkv) lds += (size_t)(BT + 1) * a.din * sizeof(uint16_t);
  lds += (size_t)(MODE == Mode::kNormQkv ? 1 : 2) * BT * ((a.rows + nblk - 1) / nblk) * sizeof(float);
  return launch_cp<BT, MAXCH, NW, NBUF, MODE>(a, grid, lds, s, ev);
}

// batch tile: as many sequences as fit `cap_bytes` of fp32 activations in LDS
template <int MAXCH, Mode MODE>
hipError_t launch_ch(const GemvArgs& a, size_t cap_bytes, hipStream_t s, KernelEvents ev) {
  const int cap = (int)(cap_bytes / ((size_t)a.din * sizeof(float)));
  const int want = a.batch < cap ? a.batch : cap;
  if constexpr (MAXCH <= 4) {  // 8 sequences only for short rows (din <= 2048)
    if (want >= 8) return launch_bt<8, MAXCH, MODE>(a, s, ev);
  }
  if (want >= 4) return launch_bt<4, MAXCH, MODE>(a, s, ev);
  if (want >= 2) return launch_bt<2, MAXCH, MODE>(a, s, ev);
  return launch_bt<1, MAXCH, MODE>(a, s, ev);
}

// rows of up to 512 chunks per lane-set are taken whole; longer ones in
// segments of 8 chunks per lane
template <Mode MODE>
hipError_t launch_mode(const GemvArgs& a, size_t cap_bytes, hipStream_t s, KernelEvents ev) {
  if ((size_t)a.din * sizeof(float) > cap_bytes) return hipErrorInvalidValue;
  const int chunks_per_lane = (a.din / 8 + kWave - 1) / kWave;
  if (chunks_per_lane <= 1) return launch_ch<1, MODE>(a, cap_bytes, s, ev);
  if (chunks_per_lane <= 2) return launch_ch<2, MODE>(a, cap_bytes, s, ev);
  if (chunks_per_lane <= 4) return launch_ch<4, MODE>(a, cap_bytes, s, ev);
  if (chunks_per_lane <= 6) return launch_ch<6, MODE>(a, cap_bytes, s, ev);
  return launch_ch<8, MODE>(a, cap_bytes, s, ev);
}

}  // namespace

// The activations of a batch tile take up to 64 KB of LDS in the attention
// projections and up to 128 KB in the down projection (its rows are K long,
// up to 32768 values).
hipError_t launch_rmsnorm_qkv(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mode<Mode::kNormQkv>(a, 65536, s, ev);
}
hipError_t launch_oproj_residual(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mode<Mode::kResidual>(a, 65536, s, ev);
}
hipError_t launch_down_residual(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mode<Mode::kDownResidual>(a, 131072, s, ev);
}

}  // namespace fasttps
