// The weight-streaming GEMV of the decode layer as a device-side body, shared
// by the one-kernel-per-projection path (gemv.hip) and the fused layer kernel
// (fused_layer.hip). See gemv.hip for the layout of the work.
//
// The body keeps its state in registers (a struct that never leaves the
// kernel) and runs in three steps:
//   load_inputs()  residuals, the activation chunks of this wave and the gains
//                  (or load_resid(), then load_act_lds() from a block's
//                  InputStage once the stage is in LDS)
//   prime()        the ring's first NBUF rows (weights do not depend on the
//                  activation, so a fused kernel primes them before it waits
//                  for the phase that produces the activation)
//   run()          the norm, the streaming loop and the segment sums
// Activations, residuals and fp32 outputs go through an IO policy: global
// memory for the separate kernels, LDS-staged inputs and agent-coherent
// stores for the fused kernel.
#pragma once

#include <math.h>

#include "common.h"
#include "kernels.h"

namespace fasttps {
namespace gemv {

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
  for (int j = 0; j < MAXCH; ++j) w[j] = ld_stream(row + min(cbase + lane + kWave * j, cmax));
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

// dot_slot for chunk j alone
template <int BT, int MAXCH>
__device__ __forceinline__ void dot_chunk(float (&acc)[BT], const v4u& w, const float (&act)[BT][MAXCH][8], int j,
                                          int nch, int cbase, int lane) {
  if (cbase + lane + kWave * j < nch) {
    float wf[8];
    unpack8(w, wf);
#pragma unroll
    for (int b = 0; b < BT; ++b) {
      float s = acc[b];
#pragma unroll
      for (int e = 0; e < 8; ++e) s = fmaf(wf[e], act[b][j][e], s);
      acc[b] = s;
    }
  }
}

// Global-memory IO of the separate kernels.
struct GlobalIO {
  // float4 i4 of activation row b
  __device__ __forceinline__ float4 act4(const GemvArgs& a, int b, int i4) const {
    return reinterpret_cast<const float4*>(a.in_f32 + (size_t)b * a.din)[i4];
  }
  __device__ __forceinline__ float res(const GemvArgs& a, size_t o) const { return a.res_f32[o]; }
  __device__ __forceinline__ void out(const GemvArgs& a, size_t o, float v) const { a.out[o] = v; }
};

template <int BT, int MAXCH, int NSEG_H, int NBUF, Mode MODE, class IO, int WAVES = kWaves>
struct GemvBody {
  static constexpr int NH = halves<MODE>();
  static constexpr int NSEG = NH * NSEG_H;
  static constexpr int NG = WAVES / NSEG;  // groups of waves
  static constexpr int kSeg = kWave * MAXCH;
  static_assert(NSEG <= WAVES && WAVES % NSEG == 0, "segments must divide the block's waves");
  static_assert(BT * MAXCH <= 6, "activation registers");

  // LDS words the body needs: part [NSEG][BT][nres] segment sums | ssq
  // [NSEG_H][BT] partial sums of squares
  static __host__ __device__ size_t lds_floats(int rows, int G) {
    return (size_t)NSEG * BT * ((rows + G - 1) / G) + (size_t)NSEG_H * BT;
  }

  const GemvArgs& a;
  IO io;
  float* part;
  float* ssq;
  int tid, lane, wave, seg, grp, half, sh, G, blk, b0, nb, nch, cbase, hoff, nres, nrow, nmine, rdead;
  size_t row_chunks;
  bool resid_reg;
  const v4u* W;
  float resid;
  float ss_in;    // staged inputs: the row's sum of squares for the norm
  bool ss_given;  // (computed by the stage, so run() does not)
  v4u xr[BT][MAXCH];        // x chunks (bf16), QKV norm mode
  float4 fr[BT][MAXCH][2];  // fp32 activation chunks, other modes
  v4u gr[MAXCH];            // gain chunks
  v4u w[NBUF][MAXCH];       // the ring

  // blk of G blocks, batch tile starting at b0; lds: lds_floats() words
  __device__ __forceinline__ GemvBody(const GemvArgs& a_, IO io_, float* lds, int blk_, int G_, int b0_, int tid_)
      : a(a_), io(io_), tid(tid_), G(G_), blk(blk_), b0(b0_) {
    lane = tid & (kWave - 1);
    wave = tid / kWave;
    seg = wave % NSEG;
    grp = wave / NSEG;
    half = seg / NSEG_H;
    sh = seg % NSEG_H;
    nb = min(BT, a.batch - b0);
    nch = a.din >> 3;  // chunks of a half row (= of the activation)
    row_chunks = (a.ld ? (size_t)a.ld : (size_t)NH * a.din) / 8;  // chunks of a stored row
    cbase = sh * kSeg;
    hoff = half * nch;
    nres = (a.rows + G - 1) / G;
    nrow = (a.rows - 1 - blk) / G + 1;  // the block's rows blk + G i, i < nrow (>= 1)
    nmine = grp < nrow ? (nrow - 1 - grp) / NG + 1 : 0;  // rows grp + NG k of this wave
    rdead = blk + G * (grp % nrow);
    // the residuals of a wave's rows fit one register per lane unless the
    // rows are many (segmented rows with large batch tiles): then run() loads
    // them at the end
    resid_reg = BT * ((nres + NG - 1) / NG) <= kWave;
    part = lds;
    ssq = lds + (size_t)NSEG * BT * nres;
    W = reinterpret_cast<const v4u*>(a.w);
    resid = 0.f;
    ss_in = 0.f;
    ss_given = false;
  }

  // ---- 1. residuals of this wave's rows, its activation chunks, the gains --
  __device__ __forceinline__ void load_inputs() {
    load_resid();
    load_act();
  }

  // residual of (b, k-th row of this wave) in lane b * nmine + k
  __device__ __forceinline__ void load_resid() {
    if (has_residual<MODE>()) {
      const int nm = nmine > 0 ? nmine : 1;
      const int q = min(lane, nb * nm - 1);
      const int qb = q / nm, qk = q % nm;
      const size_t o = (size_t)(b0 + qb) * a.rows + blk + (size_t)G * min(grp + NG * qk, nrow - 1);
      resid = MODE == Mode::kResidual ? bf16_to_f32(a.x_bf16[o]) : io.res(a, o);
    }
  }

  // the activation values of this wave's chunks, and the gains
  __device__ __forceinline__ void load_act() {
#pragma unroll
    for (int j = 0; j < MAXCH; ++j) {
      const int c = min(cbase + lane + kWave * j, nch - 1);
#pragma unroll
      for (int b = 0; b < BT; ++b) {
        const int bb = b0 + min(b, nb - 1);  // rows past the batch repeat its last one
        if (MODE == Mode::kNormQkv) {
          xr[b][j] = reinterpret_cast<const v4u*>(a.x_bf16 + (size_t)bb * a.din)[c];
        } else {
          fr[b][j][0] = io.act4(a, bb, 2 * c);
          fr[b][j][1] = io.act4(a, bb, 2 * c + 1);
        }
      }
      if (has_norm<MODE>()) gr[j] = reinterpret_cast<const v4u*>(a.gamma)[c];
    }
  }

  // the same from a block's LDS stage of one sequence (BT 1): 16-byte pieces,
  // the activation's (fp32, or bf16 x in the QKV mode) first, then the gains'
  // (wss: the stage's per-wave sums of squares, added here in wave order)
  __device__ __forceinline__ void load_act_lds(const v4u* stage, const float* wss) {
    static_assert(BT == 1, "one sequence per stage");
    const int nact = MODE == Mode::kNormQkv ? nch : 2 * nch;
    if (has_norm<MODE>()) {
      float t = 0.f;
#pragma unroll
      for (int w = 0; w < WAVES; ++w) t += wss[w];
      ss_in = t;
      ss_given = true;
    }
#pragma unroll
    for (int j = 0; j < MAXCH; ++j) {
      const int c = min(cbase + lane + kWave * j, nch - 1);
      if (MODE == Mode::kNormQkv) {
        xr[0][j] = stage[c];
      } else {
        const v4u u0 = stage[2 * c], u1 = stage[2 * c + 1];
        fr[0][j][0] = make_float4(__uint_as_float(u0.x), __uint_as_float(u0.y), __uint_as_float(u0.z),
                                  __uint_as_float(u0.w));
        fr[0][j][1] = make_float4(__uint_as_float(u1.x), __uint_as_float(u1.y), __uint_as_float(u1.z),
                                  __uint_as_float(u1.w));
      }
      if (has_norm<MODE>()) gr[j] = stage[nact + c];
    }
  }

  // ---- 2. the ring's first NBUF rows ----------------------------------------
  __device__ __forceinline__ void prime() {
#pragma unroll
    for (int k = 0; k < NBUF; ++k)
      load_slot<MAXCH>(w[k], W, row_chunks, k < nmine, blk + G * (grp + NG * k), rdead, hoff, nch, cbase, lane);
  }

  // value e of chunk j of batch row b as loaded
  __device__ __forceinline__ float src(int b, int j, int e) const {
    if (MODE == Mode::kNormQkv) return (e & 1) ? bf16_hi(xr[b][j][e >> 1]) : bf16_lo(xr[b][j][e >> 1]);
    const float4 f = fr[b][j][e >> 2];
    return (e & 3) == 0 ? f.x : (e & 3) == 1 ? f.y : (e & 3) == 2 ? f.z : f.w;
  }

  // ---- 3.-5. norm, stream this wave's rows, segment sums -------------------
  __device__ __forceinline__ void run() {
    // ---- 3. the activation in registers ------------------------------------
    float inv[BT];
#pragma unroll
    for (int b = 0; b < BT; ++b) inv[b] = 1.f;
    if (has_norm<MODE>()) {
      // RMSNorm: x / sqrt(mean(x^2) + eps) * gamma over the full row; a row
      // cut into segments adds its segments' sums of squares through LDS
      float ss[BT];
      if (ss_given) {
        // staged inputs: the stage summed the squares (uniform branch)
#pragma unroll
        for (int b = 0; b < BT; ++b) ss[b] = ss_in;
      } else {
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

    // ---- 4. stream this wave's rows ---------------------------------------
    float acc[BT];
#pragma unroll
    for (int b = 0; b < BT; ++b) acc[b] = 0.f;
    // one row in flight: the next row's chunk j goes out as soon as this
    // row's chunk j has been used (the row pointers advance by a fixed step);
    // the last row issues nothing, so nothing after the loop waits for loads
    // whose data is never used
    const v4u* rbase = W + (size_t)(blk + G * grp) * row_chunks + hoff;
    const size_t rstep = (size_t)G * NG * row_chunks;
    // the wave's k-th row is summed in acc: its outputs, or its segment's part
    auto finish = [&](int k) {
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
          else io.out(a, o, v);
        } else if (lane == 0) {
          part[((size_t)seg * BT + b) * nres + i] = v;
        }
      }
    };
    if constexpr (NBUF == 1) {
      int k = 0;
      for (; k + 1 < nmine; ++k) {
        const v4u* nrow = rbase + (size_t)(k + 1) * rstep;
#pragma unroll
        for (int j = 0; j < MAXCH; ++j) {
          dot_chunk<BT, MAXCH>(acc, w[0][j], act, j, nch, cbase, lane);
          w[0][j] = ld_stream(nrow + min(cbase + lane + kWave * j, nch - 1));
        }
        finish(k);
      }
      if (k < nmine) {
#pragma unroll
        for (int j = 0; j < MAXCH; ++j) dot_chunk<BT, MAXCH>(acc, w[0][j], act, j, nch, cbase, lane);
        finish(k);
      }
    } else {
      for (int k0 = 0; k0 < nmine; k0 += NBUF) {
#pragma unroll
        for (int s = 0; s < NBUF; ++s) {
          const int k = k0 + s;
          const bool live = k < nmine;
          if (live) dot_slot<BT, MAXCH>(acc, w[s], act, nch, cbase, lane);
          load_slot<MAXCH>(w[s], W, row_chunks, k + NBUF < nmine, blk + G * (grp + NG * (k + NBUF)), rdead, hoff,
                           nch, cbase, lane);
          if (live) finish(k);
        }
      }
    }

    // test hook: the normalized activation of this wave's chunks, written by
    // the first group's waves of the first half (after the stream, so the
    // ring's waits are not disturbed)
    if (has_norm<MODE>() && a.dbg_act && grp == 0 && half == 0 && blk == 0) {
#pragma unroll
      for (int j = 0; j < MAXCH; ++j) {
        const int c = cbase + lane + kWave * j;
        if (c < nch)
#pragma unroll
          for (int b = 0; b < BT; ++b)
            if (b < nb)
#pragma unroll
              for (int e = 0; e < 8; ++e) a.dbg_act[(size_t)(b0 + b) * a.din + (size_t)c * 8 + e] = act[b][j][e];
      }
    }

    // ---- 5. rows cut into segments: add the segments (and siLu_Mul) -------
    if (NSEG > 1) {
      __syncthreads();
      for (int t = tid; t < nb * nrow; t += WAVES * kWave) {
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
          v[0] += MODE == Mode::kResidual ? bf16_to_f32(a.x_bf16[o]) : io.res(a, o);
        if (MODE == Mode::kGateUp) io.out(a, o, v[0] / (1.0f + expf(-v[0])) * v[NH - 1]);
        else if (MODE == Mode::kDownResidual) a.out_bf16[o] = f32_to_bf16(v[0]);
        else io.out(a, o, v[0]);
      }
    }
  }
};

// The inputs of one sequence staged in LDS by the whole block: the activation
// (fp32 [din], or the token x as bf16 in the QKV mode) and the RMSNorm gains
// (bf16 [din]) as 16-byte pieces, piece p loaded by thread p mod kThreads.
// Each element then crosses the CU's load path once per block instead of
// once per wave group that uses it (the waves of a row's two halves and of
// every group of rows read the same chunks).
template <Mode MODE, int WAVES = kWaves>
struct InputStage {
  static constexpr int kThreads = WAVES * kWave;
  static constexpr int kMaxPieces = 4;  // per thread
  v4u v[kMaxPieces];
  int n, nact, per, tid;

  static __host__ __device__ int act_pieces(int din) { return MODE == Mode::kNormQkv ? din / 8 : din / 4; }
  static __host__ __device__ int pieces(int din) { return act_pieces(din) + (has_norm<MODE>() ? din / 8 : 0); }
  static __host__ __device__ bool fits(int din) { return pieces(din) <= kMaxPieces * kThreads; }

  // the loads (every one clamped to a piece that exists; `per` is uniform)
  __device__ __forceinline__ void load(const GemvArgs& a, int tid_) {
    tid = tid_;
    nact = act_pieces(a.din);
    n = pieces(a.din);
    per = (n + kThreads - 1) / kThreads;
    const v4u* act = MODE == Mode::kNormQkv ? reinterpret_cast<const v4u*>(a.x_bf16)
                                            : reinterpret_cast<const v4u*>(a.in_f32);
    const v4u* g = reinterpret_cast<const v4u*>(a.gamma);
#pragma unroll
    for (int i = 0; i < kMaxPieces; ++i)
      if (i < per) {
        const int q = min(tid + kThreads * i, n - 1);
        v[i] = has_norm<MODE>() && q >= nact ? g[q - nact] : act[q];
      }
  }

  // the pieces into the stage; for the norm modes also the sum of squares of
  // this wave's activation pieces into wss[wave] (WAVES floats of LDS)
  __device__ __forceinline__ void store(v4u* stage, float* wss) const {
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxPieces; ++i)
      if (i < per && tid + kThreads * i < n) {
        stage[tid + kThreads * i] = v[i];
        if (has_norm<MODE>() && tid + kThreads * i < nact) {
          if (MODE == Mode::kNormQkv) {
            float f[8];
            unpack8(v[i], f);
#pragma unroll
            for (int e = 0; e < 8; ++e) t = fmaf(f[e], f[e], t);
          } else {
            const float f[4] = {__uint_as_float(v[i].x), __uint_as_float(v[i].y), __uint_as_float(v[i].z),
                                __uint_as_float(v[i].w)};
#pragma unroll
            for (int e = 0; e < 4; ++e) t = fmaf(f[e], f[e], t);
          }
        }
      }
    if (has_norm<MODE>()) {
      t = wave_sum(t);
      if ((tid & (kWave - 1)) == 0) wss[tid / kWave] = t;
    }
  }
};

// Launch shape of one projection: batch tile BT, MAXCH chunks per lane and row
// segment, NSEG_H segments per half row, NBUF rows in flight per wave.
struct Shape {
  int bt, maxch, nseg_h, nbuf;
};

// Rows in flight per wave (the ring depth) for a batch tile of bt sequences
// and maxch chunks per lane: one row of 2 KB or more at one sequence and of
// 3 KB or more otherwise, else two (2-4 KB in flight per wave). At one
// sequence the Phi-3 down projection's 2 KB segments one at a time instead of
// two gave 61.1 -> 60.8 us per layer step on MI355X; two or three of the O
// projection's 3 KB segments instead of one were slower.
constexpr int ring_rows(int bt, int maxch) { return (maxch >= 3 || (bt == 1 && maxch == 2)) ? 1 : 2; }

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

}  // namespace gemv
}  // namespace fasttps
