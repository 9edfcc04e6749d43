// Weight-streaming GEMV kernels of the decode layer (gfx950): the QKV
// projection with RMSNorm1, the O projection with the residual, the fused
// gate/up projection with RMSNorm2 and siLu_Mul, and the down projection with
// the residual and the bf16 rounding of y.
//
// At batch 1-8 the projections are matrix-vector products whose cost is the
// bf16 weight stream from HBM (Section 4.4 of the paper: token-phase MLP and
// projections are bound by weight movement). Layout of the work:
//   * rows are dealt to the blocks round-robin (block b takes rows b, b + G,
//     b + 2G, ... of a grid of G blocks), so at any moment the chip reads a
//     compact window of the matrix;
//   * a row is cut into NSEG segments of 64 MAXCH 16-byte chunks; the 16
//     waves of a block form 16 / NSEG groups of NSEG waves, wave (g, s) taking
//     segment s of the group's rows g, g + 16 / NSEG, ... Lane l of a wave
//     reads chunks l, l + 64, ... of its segment, so every load instruction
//     covers one contiguous kilobyte;
//   * each wave holds the activation values of its own chunks in registers
//     (fp32), loaded before its first weight load: a wave's loads return in
//     the order they were issued, so the activation is ready as soon as the
//     first weight row is, and no wave waits for another before it computes
//     (only a row cut into segments needs the block's waves to meet: its
//     sum of squares for the norm, and its segment sums, go through LDS);
//   * each wave keeps NBUF rows in flight (2-4 KB): more outstanding loads
//     per CU only queue up in the memory system;
//   * every global load is issued unconditionally (clamped or dead addresses
//     where there is nothing to load), so the number of loads in flight is
//     the same on every path and the compiler waits for exactly the ring
//     slot a dot product needs.
// The gate/up projection reads the interlaced W_gu (Section 3.2 item 1,
// Alg. 4) with tiles of one row: row 2k is gate row k and row 2k+1 up row k,
// so one row of this kernel is the pair [gate k | up k] of 2D values, its two
// halves are the kernel's two segment halves, and siLu_Mul (Eq. 30-31)
// combines them in LDS.
#include "common.h"
#include "kernels.h"

#include <math.h>

namespace fasttps {

namespace {

// kNormQkv:      out = W RMSNorm(x)                          (x bf16; fp32 out)
// kResidual:     out = x + W act                             (x bf16, act fp32; fp32 out)
// kDownResidual: y = bf16(res + W act)                       (res, act fp32; bf16 out)
// kGateUp:       a = SiLU(W_g h) * (W_u h), h = RMSNorm(h1)  (h1 fp32; fp32 out)
// kPlain:        out = W act                                 (act fp32; fp32 out; the
//                op-by-op baseline's projections)
enum class Mode { kNormQkv, kResidual, kDownResidual, kGateUp, kPlain };

constexpr int kNumCu = 256;
constexpr int kWaves = 16;

template <Mode MODE>
constexpr int halves() { return MODE == Mode::kGateUp ? 2 : 1; }
template <Mode MODE>
constexpr bool has_norm() { return MODE == Mode::kNormQkv || MODE == Mode::kGateUp; }
template <Mode MODE>
constexpr bool has_residual() { return MODE == Mode::kResidual || MODE == Mode::kDownResidual; }

// One wave's ring slot: the 16-byte chunks cbase + lane + 64 j (j < MAXCH)
// of a half row starting at chunk hoff of row r. A chunk past the half row's
// end is clamped to its last chunk (the dot product skips it); a dead slot
// (live false) points every lane at the first chunk of row rdead, one cache
// line per instruction.
template <int MAXCH>
__device__ __forceinline__ void load_slot(v4u (&w)[MAXCH], const v4u* __restrict__ W, size_t row_chunks, bool live,
                                          int r, int rdead, int hoff, int nch, int cbase, int lane) {
  const v4u* row = W + (size_t)(live ? r : rdead) * row_chunks + (live ? hoff : 0);
  const int cmax = live ? nch - 1 : 0;
#pragma unroll
  for (int j = 0; j < MAXCH; ++j) w[j] = row[min(cbase + lane + kWave * j, cmax)];
}

template <int BT, int MAXCH>
__device__ __forceinline__ void dot_slot(float (&acc)[BT], const v4u (&w)[MAXCH], const float (&act)[BT][MAXCH][8],
                                         int nch, int cbase, int lane) {
#pragma unroll
  for (int j = 0; j < MAXCH; ++j) {
    if (cbase + lane + kWave * j < nch) {
      float wf[8];
      unpack8(w[j], wf);
#pragma unroll
      for (int b = 0; b < BT; ++b) {
        float s = acc[b];
#pragma unroll
        for (int e = 0; e < 8; ++e) s = fmaf(wf[e], act[b][j][e], s);
        acc[b] = s;
      }
    }
  }
}

template <int BT, int MAXCH, int NSEG_H, int NBUF, Mode MODE>
__global__ __launch_bounds__(kWaves * kWave) void gemv_kernel(GemvArgs a) {
  constexpr int NH = halves<MODE>();
  constexpr int NSEG = NH * NSEG_H;
  constexpr int NG = kWaves / NSEG;  // groups of waves
  constexpr int kSeg = kWave * MAXCH;
  static_assert(NSEG <= kWaves && kWaves % NSEG == 0, "segments must divide the block's waves");
  static_assert(BT * MAXCH <= 6, "activation registers");
  // LDS: part [NSEG][BT][nres] segment sums | ssq [NSEG_H][BT] partial sums of squares
  extern __shared__ __attribute__((aligned(16))) float lds[];

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int seg = wave % NSEG, grp = wave / NSEG;
  const int half = seg / NSEG_H, sh = seg % NSEG_H;
  const int G = gridDim.x, blk = blockIdx.x;
  const int b0 = blockIdx.y * BT;
  const int nb = min(BT, a.batch - b0);
  const int nch = a.din >> 3;                  // chunks of a half row (= of the activation)
  const size_t row_chunks = (a.ld ? (size_t)a.ld : (size_t)NH * a.din) / 8;  // chunks of a stored row
  const int cbase = sh * kSeg;
  const int hoff = half * nch;
  const int nres = (a.rows + G - 1) / G;
  const int nrow = (a.rows - 1 - blk) / G + 1;  // the block's rows blk + G i, i < nrow (>= 1)
  const int nmine = grp < nrow ? (nrow - 1 - grp) / NG + 1 : 0;  // rows grp + NG k of this wave
  const int rdead = blk + G * (grp % nrow);
  // the residuals of a wave's rows fit one register per lane unless the
  // rows are many (segmented rows with large batch tiles): then step 5
  // loads them
  const bool resid_reg = BT * ((nres + NG - 1) / NG) <= kWave;
  float* part = lds;
  float* ssq = lds + (size_t)NSEG * BT * nres;
  const v4u* W = reinterpret_cast<const v4u*>(a.w);

  // ---- 1. this wave's loads ahead of its weights: residuals, activation --
  // residual of (b, k-th row of this wave) in lane b * nmine + k
  float resid = 0.f;
  if (has_residual<MODE>()) {
    const int nm = nmine > 0 ? nmine : 1;
    const int q = min(lane, nb * nm - 1);
    const int qb = q / nm, qk = q % nm;
    const size_t o = (size_t)(b0 + qb) * a.rows + blk + (size_t)G * min(grp + NG * qk, nrow - 1);
    resid = MODE == Mode::kResidual ? bf16_to_f32(a.x_bf16[o]) : a.res_f32[o];
  }
  v4u xr[BT][MAXCH];        // x chunks (bf16), QKV norm mode
  float4 fr[BT][MAXCH][2];  // fp32 activation chunks, other modes
  v4u gr[MAXCH];            // gain chunks
#pragma unroll
  for (int j = 0; j < MAXCH; ++j) {
    const int c = min(cbase + lane + kWave * j, nch - 1);
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      const int bb = b0 + min(b, nb - 1);  // rows past the batch repeat its last one
      if (MODE == Mode::kNormQkv) {
        xr[b][j] = reinterpret_cast<const v4u*>(a.x_bf16 + (size_t)bb * a.din)[c];
      } else {
        const float4* src = reinterpret_cast<const float4*>(a.in_f32 + (size_t)bb * a.din) + 2 * c;
        fr[b][j][0] = src[0];
        fr[b][j][1] = src[1];
      }
    }
    if (has_norm<MODE>()) gr[j] = reinterpret_cast<const v4u*>(a.gamma)[c];
  }
  __builtin_amdgcn_sched_barrier(0);  // keep these loads ahead of the weight loads

  // ---- 2. the ring's first NBUF rows ------------------------------------
  v4u w[NBUF][MAXCH];
#pragma unroll
  for (int k = 0; k < NBUF; ++k)
    load_slot<MAXCH>(w[k], W, row_chunks, k < nmine, blk + G * (grp + NG * k), rdead, hoff, nch, cbase, lane);

  // ---- 3. the activation in registers ------------------------------------
  // value e of chunk j of batch row b as loaded
  auto src = [&](int b, int j, int e) -> float {
    if (MODE == Mode::kNormQkv) return (e & 1) ? bf16_hi(xr[b][j][e >> 1]) : bf16_lo(xr[b][j][e >> 1]);
    const float4 f = fr[b][j][e >> 2];
    return (e & 3) == 0 ? f.x : (e & 3) == 1 ? f.y : (e & 3) == 2 ? f.z : f.w;
  };
  float inv[BT];
#pragma unroll
  for (int b = 0; b < BT; ++b) inv[b] = 1.f;
  if (has_norm<MODE>()) {
    // RMSNorm: x / sqrt(mean(x^2) + eps) * gamma over the full row; a row
    // cut into segments adds its segments' sums of squares through LDS
    float ss[BT];
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      float t = 0.f;
#pragma unroll
      for (int j = 0; j < MAXCH; ++j)
        if (cbase + lane + kWave * j < nch)
#pragma unroll
          for (int e = 0; e < 8; ++e) t = fmaf(src(b, j, e), src(b, j, e), t);
      ss[b] = wave_sum(t);
    }
    if (NSEG_H > 1) {
      if (grp == 0 && half == 0 && lane == 0)
#pragma unroll
        for (int b = 0; b < BT; ++b) ssq[sh * BT + b] = ss[b];
      __syncthreads();
#pragma unroll
      for (int b = 0; b < BT; ++b) {
        float t = 0.f;
#pragma unroll
        for (int i = 0; i < NSEG_H; ++i) t += ssq[i * BT + b];
        ss[b] = t;
      }
    }
#pragma unroll
    for (int b = 0; b < BT; ++b) inv[b] = 1.0f / sqrtf(ss[b] / (float)a.din + a.eps);
  }
  float act[BT][MAXCH][8];
#pragma unroll
  for (int j = 0; j < MAXCH; ++j) {
    float g[8];
    if (has_norm<MODE>()) unpack8(gr[j], g);
#pragma unroll
    for (int b = 0; b < BT; ++b)
#pragma unroll
      for (int e = 0; e < 8; ++e) act[b][j][e] = has_norm<MODE>() ? src(b, j, e) * inv[b] * g[e] : src(b, j, e);
  }

  // ---- 4. stream this wave's rows -----------------------------------------
  float acc[BT];
#pragma unroll
  for (int b = 0; b < BT; ++b) acc[b] = 0.f;
  for (int k0 = 0; k0 < nmine; k0 += NBUF) {
#pragma unroll
    for (int s = 0; s < NBUF; ++s) {
      const int k = k0 + s;
      const bool live = k < nmine;
      if (live) dot_slot<BT, MAXCH>(acc, w[s], act, nch, cbase, lane);
      load_slot<MAXCH>(w[s], W, row_chunks, k + NBUF < nmine, blk + G * (grp + NG * (k + NBUF)), rdead, hoff, nch,
                       cbase, lane);
      if (live) {
        const int i = grp + NG * k;  // block-local row
#pragma unroll
        for (int b = 0; b < BT; ++b) {
          // batch rows past the tile's end repeat its last row, value and
          // address alike, so every store below is unconditional
          const int bs = min(b, nb - 1);
          float v = wave_sum(acc[b]);
          acc[b] = 0.f;
          if (has_residual<MODE>() && seg == 0 && resid_reg)
            v += __int_as_float(__builtin_amdgcn_readlane(__float_as_int(resid), bs * nmine + k));
          if (NSEG == 1) {
            const size_t o = (size_t)(b0 + bs) * a.rows + blk + (size_t)G * i;
            if (MODE == Mode::kDownResidual) a.out_bf16[o] = f32_to_bf16(v);
            else a.out[o] = v;
          } else if (lane == 0) {
            part[((size_t)seg * BT + b) * nres + i] = v;
          }
        }
      }
    }
  }

  // ---- 5. rows cut into segments: add the segments (and siLu_Mul) ---------
  if (NSEG > 1) {
    __syncthreads();
    for (int t = threadIdx.x; t < nb * nrow; t += blockDim.x) {
      const int b = t / nrow, i = t % nrow;
      float v[NH];
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        float s = 0.f;
#pragma unroll
        for (int q = 0; q < NSEG_H; ++q) s += part[((size_t)(h * NSEG_H + q) * BT + b) * nres + i];
        v[h] = s;
      }
      const size_t o = (size_t)(b0 + b) * a.rows + blk + (size_t)G * i;
      if (has_residual<MODE>() && !resid_reg)
        v[0] += MODE == Mode::kResidual ? bf16_to_f32(a.x_bf16[o]) : a.res_f32[o];
      if (MODE == Mode::kGateUp) a.out[o] = v[0] / (1.0f + expf(-v[0])) * v[NH - 1];
      else if (MODE == Mode::kDownResidual) a.out_bf16[o] = f32_to_bf16(v[0]);
      else a.out[o] = v[0];
    }
  }
}

// Launch shape: a batch tile of BT sequences, MAXCH chunks per lane and row
// segment, NSEG_H segments per half row, NBUF rows in flight per wave (2-4
// KB: at this size the memory system's queues stay short enough that the
// waves that start last do not finish much later than the rest).
template <int BT, int MAXCH, int NSEG_H, Mode MODE>
hipError_t launch_shape(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  constexpr int NBUF = MAXCH >= 3 ? 1 : 2;
  const int nblk = a.rows < kNumCu ? a.rows : kNumCu;
  // unsegmented rows add the residual from the register copy only
  constexpr int NG = kWaves / (halves<MODE>() * NSEG_H);
  if (halves<MODE>() * NSEG_H == 1 && has_residual<MODE>() &&
      BT * ((((a.rows + nblk - 1) / nblk) + NG - 1) / NG) > kWave)
    return hipErrorInvalidValue;
  dim3 grid(nblk, (a.batch + BT - 1) / BT);
  const size_t lds =
      ((size_t)halves<MODE>() * NSEG_H * BT * ((a.rows + nblk - 1) / nblk) + (size_t)NSEG_H * BT) * sizeof(float);
  return ext_launch(gemv_kernel<BT, MAXCH, NSEG_H, NBUF, MODE>, grid, dim3(kWaves * kWave), lds, s, ev, a);
}

template <int BT, int MAXCH, Mode MODE>
hipError_t launch_seg(const GemvArgs& a, int nseg_h, hipStream_t s, KernelEvents ev) {
  switch (nseg_h) {
    case 1: return launch_shape<BT, MAXCH, 1, MODE>(a, s, ev);
    case 2: return launch_shape<BT, MAXCH, 2, MODE>(a, s, ev);
    case 4: return launch_shape<BT, MAXCH, 4, MODE>(a, s, ev);
    case 8: return launch_shape<BT, MAXCH, 8, MODE>(a, s, ev);
    case 16:
      if constexpr (halves<MODE>() == 1) return launch_shape<BT, MAXCH, 16, MODE>(a, s, ev);
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

// Chunks per lane allowed for a batch tile: 3 (a lane's activation and ring
// stay small), or 6 for a single sequence whose rows would otherwise need
// more segments than the block has waves. BT MAXCH <= 6 keeps the lane's
// 8 BT MAXCH activation values, its ring and the loads' staging within the
// 128 registers a lane has when 16 waves share a CU.
inline int max_chunks(int bt, bool wide) { return bt == 1 ? (wide ? 6 : 3) : (bt == 2 ? (wide ? 3 : 1) : 1); }

// Segments a half row of din values needs with `maxch` chunks per lane.
inline int segments_for(int din, int maxch) {
  int n = 1;
  while (n * kWave * maxch < din / 8) n *= 2;
  return n;
}

template <int BT, Mode MODE>
hipError_t launch_bt(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  constexpr int NH = halves<MODE>();
  const int nch = a.din / 8;
  int cap = max_chunks(BT, false);
  if (segments_for(a.din, cap) * NH > kWaves) cap = max_chunks(BT, true);
  const int nseg_h = segments_for(a.din, cap);
  if (nseg_h * NH > kWaves) return hipErrorInvalidValue;
  const int per = (nch + nseg_h * kWave - 1) / (nseg_h * kWave);  // chunks per lane
  if (per <= 1) return launch_seg<BT, 1, MODE>(a, nseg_h, s, ev);
  if constexpr (BT <= 2) {
    if (per <= 2) return launch_seg<BT, 2, MODE>(a, nseg_h, s, ev);
    if (per <= 3) return launch_seg<BT, 3, MODE>(a, nseg_h, s, ev);
  }
  if constexpr (BT == 1) {
    if (per <= 4) return launch_seg<BT, 4, MODE>(a, nseg_h, s, ev);
    return launch_seg<BT, 6, MODE>(a, nseg_h, s, ev);
  }
  return hipErrorInvalidValue;
}

// batch tiles of 4, 2 or 1 sequences (the weights are read once per tile):
// the largest that the batch fills and whose segments fit the 16 waves
template <Mode MODE>
hipError_t launch_mode(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  constexpr int NH = halves<MODE>();
  if (a.batch >= 4 && segments_for(a.din, max_chunks(4, true)) * NH <= kWaves) return launch_bt<4, MODE>(a, s, ev);
  if (a.batch >= 2 && segments_for(a.din, max_chunks(2, true)) * NH <= kWaves) return launch_bt<2, MODE>(a, s, ev);
  return launch_bt<1, MODE>(a, s, ev);
}

}  // namespace

hipError_t launch_rmsnorm_qkv(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mode<Mode::kNormQkv>(a, s, ev);
}
hipError_t launch_oproj_residual(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mode<Mode::kResidual>(a, s, ev);
}
hipError_t launch_down_residual(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mode<Mode::kDownResidual>(a, s, ev);
}
hipError_t launch_gate_up(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mode<Mode::kGateUp>(a, s, ev);
}
hipError_t launch_gemv_plain(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mode<Mode::kPlain>(a, s, ev);
}

}  // namespace fasttps
