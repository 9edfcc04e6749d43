// Batched-decode projections on the matrix cores (gfx950 MFMA).
//
// With several sequences per step the four projections of the layer are
// skinny GEMMs: M = the batch, N = the output rows, K = the inputs. Their cost
// is still the bf16 weight stream from HBM, read once per step, but at 8-16
// sequences the multiply-adds (2 B per weight element and step) outgrow what
// the vector ALUs sustain next to that stream, so here they run on
// v_mfma_f32_16x16x32_bf16.
//
// Operands
//   * Weights (the MFMA B operand) are packed once into tiles of 16 output
//     rows x 32 inputs, 1 KB each, stored in the order the lanes hold them:
//     lane l keeps the 8 inputs 32 t + 8 (l / 16) .. + 7 of row 16 s + l % 16.
//     A wave's tile load is one contiguous kilobyte that lands in the
//     operand registers as it is. Tiles are stored stripe by stripe
//     (16 rows, all k-tiles), so a wave streams a contiguous run of tiles.
//     The gate/up stripe holds 8 gate rows and the 8 matching up rows (the
//     interlaced W_gu of Section 3.2 with a tile of 8 rows, Eq. 31).
//   * Activations (the A operand) are fp32. Each value v is split into two
//     bf16 levels, hi = bf16(v) and lo = bf16(v - hi), and the 16 rows of
//     the A operand are (sequence, level) pairs: row 2 i + level holds
//     sequence i of an 8-sequence batch tile. The products of bf16 weights
//     and bf16 levels are exact and accumulate in fp32; adding the two level
//     rows of the result gives W (hi + lo), within 2^-17 of W v. For the QKV
//     projection the split is exact: x * gamma1 of two bf16 numbers has at
//     most 16 significant bits, so its truncation to bf16 and the remainder
//     are both bf16 numbers and hi + lo = x * gamma1; the RMSNorm factor
//     1/rms(x) multiplies the finished sums (RMSNorm1(x) = inv * x * gamma1
//     and the projection is linear).
//   * The QKV kernel builds its operand from x and gamma1 as it streams;
//     the other three read it ready-made (split and laid out in operand
//     order) from the epilogue of the kernel before them: the attention
//     combine writes o, the O projection writes h1 * gamma2 (and per-stripe
//     sums of h1^2 for RMSNorm2), the gate/up projection writes SiLU(g) * u.
// Work split
//   * Blocks take the stripes round-robin; the 16 waves of a block split
//     the k-tiles of a stripe into 16 contiguous runs (nt tiles each, the
//     last runs padded), so a stripe's partial sums meet once, in LDS.
//   * Where the operand outweighs a block's weights, row groups of blocks
//     split the k-tiles instead and the last block of a group adds the
//     parts (split inputs, below).
//   * Each wave keeps NBUF tiles in flight (with their activation operands).
//     Every global load and store is issued unconditionally (clamped
//     addresses, duplicate stores of equal values), so the number of memory
//     operations in flight is the same on every path and the compiler waits
//     for exactly the ring slot a tile needs, also across a stripe's
//     epilogue.
#include "common.h"
#include "kernels.h"

#include <math.h>

namespace fasttps {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kMW = 16;           // waves per block
constexpr int kMT = kMW * kWave;  // threads per block
constexpr int kMGrid = 256;       // blocks (one per CU)
constexpr int kSeqTile = 8;       // sequences per MFMA (two levels each)
constexpr int kGroupSeq = 16;     // sequences per block row of the grid (two batch tiles)
constexpr int kMaxStripesIn = 1024;  // stripes of the O projection's sums of squares (D <= 8192 at 8 rows)
// LDS for the partial sums of one chunk of stripes: every chunk ends in a
// block barrier, so a chunk holds all of a block's stripes where it can (four
// at 16 sequences). With 40 KB the 16-sequence Phi-3 layer's QKV (3 stripes
// per block) and gate/up (4) projections met at a barrier mid-stream: on
// MI355X 64 KB gave QKV 15.9 -> 14.3 us, gate/up 21.4 -> 20.3 us and the
// layer step 148 -> 144 us
constexpr int kMaxChunkBytes = 64 * 1024;
constexpr int kMaxHidden = 8192;           // inputs of the QKV projection (gamma1 in LDS)
constexpr int kMaxParts = 4;               // input parts of a split projection

enum class MMode { kQkv, kOproj, kGateUp, kDown };

__device__ __forceinline__ bf16x8 as_bf16x8(v4u v) { return __builtin_bit_cast(bf16x8, v); }

// bf16 bits of a float, nearest even, as selects (no branches in the
// streaming loop); NaN stays a quiet NaN
__device__ __forceinline__ uint32_t bf16_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t r = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
  return f != f ? ((u >> 16) | 0x40u) : r;
}

// level `lvl` of the same split, selected per element (the form of the
// widest cached runs, whose registers the lean form below does not fit)
__device__ __forceinline__ v4u split8_exact_sel(const float (&v)[8], int lvl) {
  uint32_t h[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t u = __float_as_uint(v[j]);
    h[j] = lvl ? __float_as_uint(v[j] - __uint_as_float(u & 0xFFFF0000u)) >> 16 : u >> 16;
  }
  return v4u{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
}

// One level of the exact split of 8 values of at most 16 significant bits
// (products of two bf16 numbers), chosen by the mask m of the lane's level:
// with m = 0 the value stays, and its top half is hi, its truncation to bf16;
// with m = 0xFFFF0000 the truncation is subtracted, leaving lo = v - hi, which
// has at most 8 significant bits, so its top half is a bf16 number too and
// hi + lo = v. The top halves of two words pack with one byte permute.
__device__ __forceinline__ v4u split8_exact(const float (&v)[8], uint32_t m) {
  uint32_t t[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) t[j] = __float_as_uint(v[j] - __uint_as_float(__float_as_uint(v[j]) & m));
  return v4u{__builtin_amdgcn_perm(t[1], t[0], 0x07060302u), __builtin_amdgcn_perm(t[3], t[2], 0x07060302u),
             __builtin_amdgcn_perm(t[5], t[4], 0x07060302u), __builtin_amdgcn_perm(t[7], t[6], 0x07060302u)};
}

// element offset of (sequence b, input k, level) in an operand buffer of
// nbtc batch tiles: [k-tile][batch tile][lane][8]
__device__ __forceinline__ size_t operand_offset(int b, int k, int lvl, int nbtc) {
  const int t = k >> 5, kg = (k >> 3) & 3, j = k & 7;
  const int bt = b / kSeqTile, bp = b % kSeqTile;
  const int lane = 2 * bp + lvl + 16 * kg;
  return (((size_t)t * nbtc + bt) * kWave + lane) * 8 + j;
}

// One wave's share of the streaming: its k-tiles [tbase, tbase + nt) of every
// stripe of the block. NT > 0: the operands of those NT k-tiles are built
// once and held in registers (acache), and the ring carries weight tiles only
// (NT % NBUF == 0, so ring slots are static across stripes). NT == 0: the
// ring carries each tile's operands with it (inputs too wide to cache; such
// a matrix has few stripes per block, so little would be reused).
template <MMode MODE, int NBT, int NT, int NBUF>
__global__ __launch_bounds__(kMT) void mfma_proj_kernel(MfmaArgs a) {
  constexpr bool CACHED = NT > 0;
  constexpr int NOUT = NBT * kSeqTile * 16;  // (sequence, column) slots of a stripe
  static_assert(kMT % NOUT == 0, "epilogue slots");
  static_assert(!CACHED || NT % NBUF == 0, "static ring slots");
  extern __shared__ float red[];                // [a.sch][kMW][NOUT]: per wave, level-summed
  __shared__ float ssq[kMW][NBT * kSeqTile];    // per-wave sums of squares (QKV, gate/up)
  __shared__ v4u gam[MODE == MMode::kQkv ? kMaxHidden / 8 : 1];  // QKV: gamma1

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // uniform: scalar loop control
  const int G = gridDim.x, blk = blockIdx.x;
  // split inputs: block blk is part kq of row group rg; the ks blocks of a
  // group take the same stripes over disjoint ranges of k-tiles
  const int ks = a.ks;
  const int rg = blk / ks, kq = blk - rg * ks;
  const int NGr = G / ks;                             // row groups
  const int b0 = blockIdx.y * kGroupSeq;              // first sequence of this grid row
  const int nb = min(NBT * kSeqTile, a.batch - b0);   // sequences of this grid row
  const int nstr = (a.ns - 1 - rg) / NGr + 1;         // stripes rg, rg + NGr, ... (>= 1)
  const int nt = CACHED ? NT : a.nt;
  const int ntp = CACHED ? NT : (nt + NBUF - 1) / NBUF * NBUF;
  const int kbeg = kq * a.ktq, kend = min(kbeg + a.ktq, a.kt);  // this part's k-tiles
  const int tbase = kbeg + wave * nt;
  const int R = a.rh;                                  // rows per stripe (<= 16)
  const int n16 = lane & 15, kg = lane >> 4;
  const int bp = n16 >> 1, lvl = lane & 1;
  const int btg0 = b0 / kSeqTile;                     // first batch tile of this grid row
  const v4u* W = reinterpret_cast<const v4u*>(a.w);
  // operand lane whose data this lane loads: a sequence slot past the batch
  // reads the last sequence's (its result rows are discarded), so a partly
  // filled tile moves only its real rows
  auto op_lane = [&](int bt) {
    const int last = max(min(kSeqTile, nb - bt * kSeqTile), 1) - 1;
    return 2 * min(bp, last) + lvl + 16 * kg;
  };

  // ---- gate/up: RMSNorm2's sums of squares from the O projection ----------
  float ssq_pre = 0.f;
  if (MODE == MMode::kGateUp) {
    constexpr int PER = kMaxStripesIn / (kMT / 16);
    const int bq = min(tid % 16, nb - 1), sq = tid / 16;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int s = sq + (kMT / 16) * i;
      const float v = a.ssq_in[(size_t)min(s, a.ns_in - 1) * a.batch + b0 + bq];
      ssq_pre += s < a.ns_in ? v : 0.f;
    }
  }

  // The QKV operand of one k-tile and batch tile: x * gamma1 of this lane's
  // chunk (exact: two bf16 factors), split into the lane's level; s2: the
  // chunk's sum of x^2. gamma1 comes zero past the matrix (gamma_tile), so
  // those products are zero; the caller drops their sums of squares.
  // Sequence slots past the batch hold the last sequence's x, and no
  // epilogue reads their rows.
  // The lean form runs wherever the registers allow it: on MI355X it took the
  // 16-sequence Phi-3 QKV projection from 14.2 to 13.6 us (the build is most
  // of that kernel's vector work); with two batch tiles and runs of 7 or 8
  // cached k-tiles it spilled inside the stripe loop (16-sequence GQA shape:
  // 15.6 -> 17.5 us), so those keep the per-element form (qkv_operand_sel).
  constexpr bool LEAN = !(NBT == 2 && NT >= 7);
  const uint32_t lvmask = lvl ? 0xFFFF0000u : 0u;
  auto qkv_operand = [&](v4u xv, v4u gv, float& s2) -> v4u {
    float xf[8], g[8], v[8];
    unpack8(xv, xf);
    unpack8(gv, g);
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      v[e] = xf[e] * g[e];
      s = fmaf(xf[e], xf[e], s);
    }
    s2 = s;
    return split8_exact(v, lvmask);
  };
  auto x_chunk = [&](int t, int bt) {
    const int k0 = min(32 * min(t, a.kt - 1) + 8 * kg, a.din - 8);
    const int b = b0 + min(bt * kSeqTile + bp, nb - 1);
    return *reinterpret_cast<const v4u*>(a.x_bf16 + (size_t)b * a.din + k0);
  };
  auto g_chunk = [&](int t) {  // from the LDS copy (this wave's entries)
    const int k0 = min(32 * min(t, a.kt - 1) + 8 * kg, a.din - 8);
    return gam[k0 / 8];
  };
  // the per-element form: zero past the matrix or the batch; ss: the lane's
  // sum of x^2 (level-0 lanes, real entries; else 0)
  auto qkv_operand_sel = [&](v4u xv, v4u gv, int t, int bt, float& ss) -> v4u {
    float xf[8], g[8], v[8];
    unpack8(xv, xf);
    unpack8(gv, g);
    const bool ok = t < a.kt && 32 * t + 8 * kg < a.din && bt * kSeqTile + bp < nb;
    float s2 = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      v[e] = ok ? xf[e] * g[e] : 0.f;
      s2 = fmaf(xf[e], xf[e], s2);
    }
    ss = ok && lvl == 0 ? s2 : 0.f;
    return split8_exact_sel(v, lvl);
  };
  // gamma1 of k-tile t for this lane's k-group, zero past the matrix; ok:
  // whether the chunk is inside it
  auto gamma_tile = [&](int t, bool& ok) {
    ok = t < a.kt && 32 * t + 8 * kg < a.din;
    const v4u z = {0u, 0u, 0u, 0u};
    return ok ? g_chunk(t) : z;
  };
  // QKV with two batch tiles: the two level lanes of a (sequence slot,
  // k-group) need the same x chunks, so lane level l loads batch tile l's and
  // the pair swaps them (one load per k-tile instead of two)
  constexpr bool XPAIR = MODE == MMode::kQkv && CACHED && NBT == 2 && NT <= 6;  // (runs of 8 tiles: spills)
  // with one batch tile, the level lanes load two consecutive k-tiles of the
  // same sequence slot instead and swap them (one load per two k-tiles)
  constexpr bool XPAIR1 = MODE == MMode::kQkv && CACHED && NBT == 1 && NT % 2 == 0;
  // ready operands of at most four sequences (one batch tile): the lanes of
  // slots 4..7 load the next k-tile's slots 0..3 instead, so one load brings
  // two k-tiles (row rotation by 8 hands them to the lanes of slots 0..3)
  const bool apack = MODE != MMode::kQkv && CACHED && NBT == 1 && NT % 2 == 0 && nb <= kSeqTile / 2;
  auto packed_chunk = [&](int t) {
    const bool hi = bp >= kSeqTile / 2;
    const int slot = min(hi ? bp - kSeqTile / 2 : bp, nb - 1);
    const int tt = min(hi ? t + 1 : t, a.kt - 1);
    return reinterpret_cast<const v4u*>(a.a_in)[((size_t)tt * a.nbtc + btg0) * kWave + 2 * slot + lvl + 16 * kg];
  };
  auto ready_chunk = [&](int t, int bt) {
    return reinterpret_cast<const v4u*>(a.a_in)[((size_t)min(t, a.kt - 1) * a.nbtc + btg0 + bt) * kWave + op_lane(bt)];
  };

  float ssp[NBT];  // QKV: this lane's sums of x^2
#pragma unroll
  for (int bt = 0; bt < NBT; ++bt) ssp[bt] = 0.f;

  // ---- loads issued ahead of the weight stream: gamma1 (QKV), the cached
  // operands (or the x chunks they are built from)
  // QKV: each wave stages the gamma1 chunks of its own k-tiles (lane 4 tt +
  // k-group; a run has at most 16 tiles), so no block barrier waits for the
  // other waves' loads; lanes past the run write a neighbour's entries with
  // the values it writes itself
  const int gk8 = min(32 * min(tbase + lane / 4, a.kt - 1) + 8 * (lane & 3), a.din - 8) / 8;
  v4u gload = {0u, 0u, 0u, 0u};
  if (MODE == MMode::kQkv) gload = reinterpret_cast<const v4u*>(a.gamma)[gk8];
  v4u acache[CACHED ? NT : 1][NBT];
  if constexpr (CACHED) {
#pragma unroll
    for (int tt = 0; tt < NT; ++tt) {
      if constexpr (XPAIR) {
        acache[tt][0] = x_chunk(tbase + tt, lvl);
      } else if constexpr (XPAIR1) {
        if (tt % 2 == 0) acache[tt][0] = x_chunk(tbase + tt + lvl, 0);
      } else if (apack) {
        if (tt % 2 == 0) acache[tt][0] = packed_chunk(tbase + tt);
      } else {
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt)
          acache[tt][bt] = MODE == MMode::kQkv ? x_chunk(tbase + tt, bt) : ready_chunk(tbase + tt, bt);
      }
    }
  }
  __builtin_amdgcn_sched_barrier(0);

  // ---- the ring: item j = (stripe j / ntp, k-tile tbase + j % ntp) -------
  v4u wr[NBUF];
  v4u ar[CACHED ? 1 : NBUF][NBT];  // streamed: ready operand, or (QKV) the x chunk
  auto load_item = [&](int r, int j) {
    const int si = min(j / ntp, nstr - 1);
    const int t = min(tbase + j % ntp, kend - 1);
    const int s = rg + si * NGr;
    wr[r] = ld_stream(W + (((size_t)s * a.kt + t) * 4 + kg) * R + min(n16, R - 1));
    if constexpr (!CACHED) {
      if (MODE == MMode::kQkv) {
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) ar[r][bt] = x_chunk(t, bt);
      } else {
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) ar[r][bt] = ready_chunk(t, bt);
      }
    }
  };
  // in slot order: a wave's loads return in issue order, so slot 0 must be
  // the oldest for the loop to wait for one slot at a time
#pragma unroll
  for (int r = 0; r < NBUF; ++r) {
    load_item(r, r);
    __builtin_amdgcn_sched_barrier(0);
  }
  // gamma1 into LDS (its load is the oldest, so this waits for it only);
  // read back by this wave only, so no barrier
  if (MODE == MMode::kQkv) gam[gk8] = gload;
  // the cached operands, once their loads (older than the ring's) are in;
  // the QKV operands are built from their x chunks during the first stripe
  // instead, each just before its first MFMA, where the conversion overlaps
  // the weight stream (built here, all at once, it held the stream ~4 us)
  if constexpr (CACHED && MODE != MMode::kQkv) {
    const v4u z = {0u, 0u, 0u, 0u};
    if (apack) {
      if constexpr (NBT == 1 && NT % 2 == 0) {
#pragma unroll
        for (int tt = 0; tt < NT; tt += 2) {
          const v4u raw = acache[tt][0];
          const v4u nxt = v4u{__float_as_uint(dpp_mov<kDppRowRor8>(__uint_as_float(raw.x))),
                              __float_as_uint(dpp_mov<kDppRowRor8>(__uint_as_float(raw.y))),
                              __float_as_uint(dpp_mov<kDppRowRor8>(__uint_as_float(raw.z))),
                              __float_as_uint(dpp_mov<kDppRowRor8>(__uint_as_float(raw.w)))};
          const bool lo = bp < kSeqTile / 2;
          acache[tt][0] = lo ? raw : z;
          acache[tt + 1][0] = lo ? nxt : z;
        }
      }
    }
#pragma unroll
    for (int tt = 0; tt < NT; ++tt)
#pragma unroll
      for (int bt = 0; bt < NBT; ++bt) acache[tt][bt] = tbase + tt < kend ? acache[tt][bt] : z;
  }
  if (MODE == MMode::kGateUp) {
    // the wave's share of RMSNorm2's sums (loads issued first, so this waits
    // for them only)
    float v = ssq_pre;
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    if (lane < NBT * kSeqTile) ssq[wave][lane] = v;
  }

  // ---- stream the stripes; partial sums go to LDS, summed per chunk ------
  float inv = 1.f;  // the norm factor of this thread's epilogue sequence
  int c0 = 0;       // first stripe of the current chunk
  constexpr int NCOL = 16;
  // RMSNorm's factor for this thread's epilogue sequence, from the per-wave
  // sums of squares in LDS
  auto norm_factor = [&]() {
    const int bl = min(tid % NOUT / NCOL, nb - 1);
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < kMW; ++w) t += ssq[w][bl];
    return 1.0f / sqrtf(t / (float)a.din + a.eps);
  };
  // the mode's epilogue for slot o (sequence o / NCOL, column o % NCOL) of
  // stripe s; col(cc) is the finished sum of column cc for that sequence
  auto finish = [&](int s, int o, auto col) {
    const int bl = min(o / NCOL, nb - 1);
    const int b = b0 + bl;
    if (MODE == MMode::kGateUp) {
      const int U = R / 2;  // units per stripe: gate columns [0, U), up columns [U, 2U)
      const int nreal = min(U, a.rows - U * s);
      const int n = min(o % NCOL, nreal - 1);
      const int u = U * s + n;
      const float gt = inv * col(n), up = inv * col(n + U);
      const float av = gt / (1.0f + expf(-gt)) * up;
      a.out[(size_t)b * a.rows + u] = av;
      const uint32_t hi = bf16_bits(av);
      const uint32_t lo = bf16_bits(av - __uint_as_float(hi << 16));
      a.a_out[operand_offset(b, u, 0, a.a_out_nbtc)] = (uint16_t)hi;
      a.a_out[operand_offset(b, u, 1, a.a_out_nbtc)] = (uint16_t)lo;
    } else {
      const int nreal = min(R, a.rows - R * s);
      const int n = min(o % NCOL, nreal - 1);
      const int row = R * s + n;
      const size_t oi = (size_t)b * a.rows + row;
      if (MODE == MMode::kQkv) {
        a.out[oi] = inv * col(n);
      } else if (MODE == MMode::kOproj) {
        const float h1 = bf16_to_f32(a.x_bf16[oi]) + col(n);
        a.out[oi] = h1;
        // the gate/up operand: split of h1 * gamma2 at input `row`
        const float hg = h1 * bf16_to_f32(a.gamma[row]);
        const uint32_t hi = bf16_bits(hg);
        const uint32_t lo = bf16_bits(hg - __uint_as_float(hi << 16));
        a.a_out[operand_offset(b, row, 0, a.a_out_nbtc)] = (uint16_t)hi;
        a.a_out[operand_offset(b, row, 1, a.a_out_nbtc)] = (uint16_t)lo;
        // this stripe's sum of h1^2 per sequence (the 16 columns are one DPP row)
        float sq = o % NCOL < nreal ? h1 * h1 : 0.f;
        sq = row_stride4_sum(quad_sum(sq));
        a.ssq_out[(size_t)s * a.batch + b] = sq;
      } else {
        a.out_bf16[oi] = f32_to_bf16(a.res_f32[oi] + col(n));
      }
    }
  };
  // split inputs: this block's partial sums [stripe][slot]
  float* kp_own = ks > 1 ? a.kpart + ((size_t)blockIdx.y * G + blk) * a.kstride : nullptr;
  // stripe si (its partial sums into LDS; the epilogue after the last stripe
  // of a chunk)
  // LAST (the block's last stripe): refill only items of this stripe; the
  // refills past it would be clamped loads that nothing uses, and the
  // epilogue would wait for them (it reuses their registers)
  auto stripe = [&](int si, auto last_tag) {
    constexpr bool LAST = decltype(last_tag)::value;
    f4 acc[NBT];
#pragma unroll
    for (int bt = 0; bt < NBT; ++bt) acc[bt] = f4{0.f, 0.f, 0.f, 0.f};
    for (int tt0 = 0; tt0 < ntp; tt0 += NBUF) {
#pragma unroll
      for (int r = 0; r < NBUF; ++r) {
        const int tt = tt0 + r;
        bf16x8 A[NBT];
        if constexpr (CACHED) {
          if constexpr (XPAIR) {
            if (si == 0) {
              const v4u own = acache[tt][0], other = dpp_swap_pair(own);
              acache[tt][1] = lvl ? own : other;
              acache[tt][0] = lvl ? other : own;
            }
          } else if constexpr (XPAIR1) {
            if (si == 0 && tt % 2 == 0) {
              const v4u own = acache[tt][0], other = dpp_swap_pair(own);
              acache[tt + 1][0] = lvl ? own : other;
              acache[tt][0] = lvl ? other : own;
            }
          }
          if constexpr (LEAN) {
            if (MODE == MMode::kQkv && si == 0) {
              bool gok;
              const v4u g = gamma_tile(tbase + tt, gok);
#pragma unroll
              for (int bt = 0; bt < NBT; ++bt) {
                float s2;
                acache[tt][bt] = qkv_operand(acache[tt][bt], g, s2);
                ssp[bt] += gok ? s2 : 0.f;
              }
            }
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) A[bt] = as_bf16x8(acache[tt][bt]);
          } else {
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) {
              if (MODE == MMode::kQkv && si == 0) {
                float s2;
                acache[tt][bt] = qkv_operand_sel(acache[tt][bt], g_chunk(tbase + tt), tbase + tt, bt, s2);
                ssp[bt] += s2;
              }
              A[bt] = as_bf16x8(acache[tt][bt]);
            }
          }
        } else {
          const int t = tbase + tt;
          const bool live = tt < nt && t < kend;
          if (MODE == MMode::kQkv) {
            bool gok;
            const v4u g = gamma_tile(live ? t : a.kt, gok);
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) {
              float s2;
              A[bt] = as_bf16x8(qkv_operand(ar[r][bt], g, s2));
              if (si == 0) ssp[bt] += gok ? s2 : 0.f;
            }
          } else {
            // a padding item (past the wave's run or the matrix) adds zero
            const v4u z = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int bt = 0; bt < NBT; ++bt) A[bt] = as_bf16x8(live ? ar[r][bt] : z);
          }
        }
        const bf16x8 B = as_bf16x8(wr[r]);
#pragma unroll
        for (int bt = 0; bt < NBT; ++bt) acc[bt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[bt], B, acc[bt], 0, 0, 0);
        // refill the slot with the item NBUF further on (clamped past the end);
        // the barrier keeps the refill after the MFMAs, so the new tile lands
        // in the registers the old one leaves (no copies, no early waits)
        __builtin_amdgcn_sched_barrier(0);
        if (!LAST || tt + NBUF < ntp) load_item(r, si * ntp + tt + NBUF);
      }
    }

    // lane l holds rows 4 (l / 16) + i of the result: sequences 2 (l / 16)
    // and 2 (l / 16) + 1 of each tile, the two levels in register pairs
    float* rw = red + ((size_t)(si - c0) * kMW + wave) * NOUT;
#pragma unroll
    for (int bt = 0; bt < NBT; ++bt) {
      const int q0 = (bt * kSeqTile + 2 * kg) * 16 + n16;
      rw[q0] = acc[bt][0] + acc[bt][1];
      rw[q0 + 16] = acc[bt][2] + acc[bt][3];
    }
    if (MODE == MMode::kQkv && si == 0) {
      // the wave's sums of x^2 per sequence: level-0 lanes of the four k groups
#pragma unroll
      for (int bt = 0; bt < NBT; ++bt) {
        float v = ssp[bt];
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        if (lane < 16 && lvl == 0) ssq[wave][bt * kSeqTile + bp] = v;
      }
    }
    if (si - c0 + 1 < a.sch && si + 1 < nstr) return;

    // ---- epilogue of stripes c0 .. si -------------------------------------
    __syncthreads();
    const int nch = si - c0 + 1;
    // thread tid serves slot tid % NOUT of stripes c0 + tid / NOUT, ... (a
    // uniform count of rounds, stripes clamped into the chunk, sequences
    // past the batch and columns past the matrix clamped to real ones, so
    // every store is unconditional and duplicates store equal values)
    const int o = tid % NOUT;
    const int rounds = (a.sch * NOUT + kMT - 1) / kMT;
    if (MODE != MMode::kQkv && ks > 1) {
      // this part's sums of the chunk's stripes, for the group's last block
      for (int rd = 0; rd < rounds; ++rd) {
        const int c = min((tid + rd * kMT) / NOUT, nch - 1);
        const float* rc = red + (size_t)c * kMW * NOUT;
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < kMW; ++w) v += rc[w * NOUT + o];
        st_c(kp_own + (size_t)(c0 + c) * NOUT + o, v);
      }
    } else {
      if ((MODE == MMode::kQkv || MODE == MMode::kGateUp) && c0 == 0) inv = norm_factor();
      const int bl = min(o / NCOL, nb - 1);
      for (int rd = 0; rd < rounds; ++rd) {
        const int c = min((tid + rd * kMT) / NOUT, nch - 1);
        const float* rc = red + (size_t)c * kMW * NOUT + bl * NCOL;
        finish(rg + (c0 + c) * NGr, o, [&](int cc) {
          float v = 0.f;
#pragma unroll
          for (int w = 0; w < kMW; ++w) v += rc[w * NOUT + cc];
          return v;
        });
      }
    }
    __syncthreads();
    c0 = si + 1;
  };
  // (the widest cached runs with two batch tiles keep one stripe body: a
  // second copy of it spills there)
  if constexpr (NBT == 2 && NT >= 7) {
    for (int si = 0; si < nstr; ++si) stripe(si, BoolTag<false>{});
  } else {
    for (int si = 0; si + 1 < nstr; ++si) stripe(si, BoolTag<false>{});
    stripe(nstr - 1, BoolTag<true>{});
  }

  // ---- split inputs: the group's last block sums the parts in order -------
  if constexpr (MODE != MMode::kQkv) {
    if (ks > 1) {
      __shared__ int last_part;
      wait_vm();  // this block's partial sums are stored
      __syncthreads();
      if (tid == 0) {
        unsigned* tk = a.tickets + (size_t)blockIdx.y * NGr + rg;
        const unsigned prev = __hip_atomic_fetch_add(tk, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const bool lst = prev == (unsigned)(ks - 1);
        if (lst) st_cu(tk, 0u);  // ready for the next launch
        last_part = lst;
      }
      __syncthreads();
      if (!last_part) return;
      if (MODE == MMode::kGateUp) inv = norm_factor();
      const float* kp_grp = a.kpart + ((size_t)blockIdx.y * G + rg * ks) * a.kstride;
      const int o = tid % NOUT;
      const int bl = min(o / NCOL, nb - 1);
      const int rounds = (nstr * NOUT + kMT - 1) / kMT;
      for (int rd = 0; rd < rounds; ++rd) {
        const int c = min((tid + rd * kMT) / NOUT, nstr - 1);
        const float* pc = kp_grp + (size_t)c * NOUT + bl * NCOL;
        finish(rg + c * NGr, o, [&](int cc) {
          float v = 0.f;
#pragma unroll
          for (int q = 0; q < kMaxParts; ++q)
            if (q < ks) v += ld_c(pc + (size_t)q * a.kstride + cc);
          return v;
        });
      }
    }
  }
}

template <MMode MODE, int NBT>
hipError_t launch_nbt(const MfmaArgs& a, int ngr, hipStream_t s, KernelEvents ev) {
  dim3 grid(ngr * a.ks, (a.batch + kGroupSeq - 1) / kGroupSeq);
  const size_t lds = (size_t)a.sch * kMW * NBT * kSeqTile * 16 * sizeof(float);
  const int nt = a.nt;
  // operands cached when the wave's run is short enough for its registers;
  // the whole run in flight at once (measured: 16-sequence Phi-3 and 4 x
  // 32768 GQA layers ~1.5 us faster each than with half of it), except the
  // 16-sequence QKV kernel with 8 tiles, which would spill
  if (nt <= 8 && nt * NBT <= 16) {
    switch (nt) {
      case 1: return ext_launch(mfma_proj_kernel<MODE, NBT, 1, 1>, grid, dim3(kMT), lds, s, ev, a);
      case 2: return ext_launch(mfma_proj_kernel<MODE, NBT, 2, 2>, grid, dim3(kMT), lds, s, ev, a);
      case 3: return ext_launch(mfma_proj_kernel<MODE, NBT, 3, 3>, grid, dim3(kMT), lds, s, ev, a);
      case 4: return ext_launch(mfma_proj_kernel<MODE, NBT, 4, 4>, grid, dim3(kMT), lds, s, ev, a);
      case 5: return ext_launch(mfma_proj_kernel<MODE, NBT, 5, 5>, grid, dim3(kMT), lds, s, ev, a);
      case 6: return ext_launch(mfma_proj_kernel<MODE, NBT, 6, 6>, grid, dim3(kMT), lds, s, ev, a);
      case 7: return ext_launch(mfma_proj_kernel<MODE, NBT, 7, 7>, grid, dim3(kMT), lds, s, ev, a);
      default:
        if constexpr (MODE == MMode::kQkv && NBT == 2)
          return ext_launch(mfma_proj_kernel<MODE, NBT, 8, 4>, grid, dim3(kMT), lds, s, ev, a);
        else
          return ext_launch(mfma_proj_kernel<MODE, NBT, 8, 8>, grid, dim3(kMT), lds, s, ev, a);
    }
  }
  if (nt % 4 == 0) return ext_launch(mfma_proj_kernel<MODE, NBT, 0, 4>, grid, dim3(kMT), lds, s, ev, a);
  if (nt % 3 == 0) return ext_launch(mfma_proj_kernel<MODE, NBT, 0, 3>, grid, dim3(kMT), lds, s, ev, a);
  return ext_launch(mfma_proj_kernel<MODE, NBT, 0, 2>, grid, dim3(kMT), lds, s, ev, a);
}

// stripes of the block whose partial sums share LDS before one epilogue
inline int chunk_stripes(int per_block, int nbt) {
  const int cap = kMaxChunkBytes / (kMW * nbt * kSeqTile * 16 * (int)sizeof(float));
  return per_block < cap ? per_block : cap;
}

// Split inputs. Every block reads the whole activation operand of its k-tiles
// (4 bytes per input and sequence, two bf16 levels: nbt KB per k-tile), and
// a CU serves those loads in the same queue as its weight stream, so where
// the operand outweighs a block's weights it costs more time than they do
// (the down projection of the 16-sequence Phi-3 layer: 512 KB of operand
// against 196 KB of weights per block). There the k-tiles are split into
// kSplit parts: a row group of kSplit blocks takes the same stripes, each
// block one part, so a block holds kSplit times the stripes and a kSplit-th
// of the operand. Each block stores its partial sums (coherent stores), then
// takes a ticket of its group; the last block of the group adds the partial
// sums in part order and runs the epilogue, so the result does not depend on
// which block comes last. The tickets and the last block's loads add about
// 1.5 us, so the split is taken only where the operand is at least twice a
// block's weights and 256 KB or more. Measured on MI355X (kernel us, split
// into 4 against whole rows): 16-sequence Phi-3 down 19.1 -> 14.3 (taken);
// its O projection (196 KB of operand) 8.4 -> 9.9 and gate/up (in 2 parts,
// operand half the weights) 21.8 -> 22.9; GQA layer at 4 sequences (operand
// equal to the weights) O 11.0 -> 10.2, down 21.6 -> 23.8.
constexpr int kSplit = 4;
constexpr int kSplitMinTiles = 128;     // k-tiles: 128 nbt KB of operand
constexpr int kMinPartTiles = kMW / 2;  // k-tiles per part at least (half the waves busy)

int nbt_of(int batch) { return batch > kSeqTile ? 2 : 1; }

struct SplitGeom {
  int ks, ngr, ktq, nt, nstr_max;
};
SplitGeom split_geom(MMode mode, int ns, int kt, int rh, int nbt) {
  const int nstr0 = (ns + kMGrid - 1) / kMGrid;  // stripes per block, whole rows
  // operand bytes (nbt KB per k-tile) >= 2 x weight bytes (rh x 64 B per k-tile and stripe)
  const bool heavy = 16 * nbt >= 2 * nstr0 * rh && kt >= kSplitMinTiles;
  int ks = mode != MMode::kQkv && heavy ? kSplit : 1;
  while (ks > 1 && (kt < ks * kMinPartTiles || (ks - 1) * ((kt + ks - 1) / ks) >= kt)) ks /= 2;
  SplitGeom g;
  g.ks = ks;
  g.ngr = ns < kMGrid / ks ? ns : kMGrid / ks;
  g.ktq = (kt + ks - 1) / ks;
  g.nt = (g.ktq + kMW - 1) / kMW;
  g.nstr_max = (ns + g.ngr - 1) / g.ngr;
  return g;
}

template <MMode MODE>
hipError_t launch_mmode(const MfmaArgs& a_in, hipStream_t s, KernelEvents ev) {
  MfmaArgs a = a_in;
  if (a.batch < 1 || a.ns < 1 || a.kt < 1 || a.nt != (a.kt + kMW - 1) / kMW || a.din % 8 != 0) return hipErrorInvalidValue;
  if (MODE == MMode::kQkv && a.din > kMaxHidden) return hipErrorInvalidValue;  // gamma1 in LDS, 16 tiles per wave
  if (a.rh < 2 || a.rh > 16 || a.rh % 2 != 0) return hipErrorInvalidValue;
  if (MODE == MMode::kGateUp && a.ns_in > kMaxStripesIn) return hipErrorInvalidValue;
  const int nbt = nbt_of(a.batch);
  SplitGeom g = split_geom(MODE, a.ns, a.kt, a.rh, nbt);
  const size_t nout = (size_t)nbt * kSeqTile * 16;
  const size_t ny = (a.batch + kGroupSeq - 1) / kGroupSeq;
  if (g.ks > 1 && (!a.kpart || !a.tickets || a.kpart_cap < ny * g.ngr * g.ks * g.nstr_max * nout ||
                   a.tickets_cap < ny * g.ngr)) {
    g.ks = 1;  // no scratch for the parts: whole rows per block
    g.ngr = a.ns < kMGrid ? a.ns : kMGrid;
    g.ktq = a.kt;
    g.nt = a.nt;
    g.nstr_max = (a.ns + g.ngr - 1) / g.ngr;
  }
  a.ks = g.ks;
  a.ktq = g.ktq;
  a.nt = g.nt;
  a.kstride = (int)(g.nstr_max * nout);
  a.sch = chunk_stripes(g.nstr_max, nbt);
  if (nbt == 2) return launch_nbt<MODE, 2>(a, g.ngr, s, ev);
  return launch_nbt<MODE, 1>(a, g.ngr, s, ev);
}

// Tiled copy of a row-major [rows, din] matrix (stride ld elements) in
// stripes of R rows: tile (s, t) holds, for k-group kg and row n < R, the 16
// bytes of row R s + n at inputs 32 t + 8 kg .. + 7, at chunk
// ((s kt + t) 4 + kg) R + n; zero outside the matrix. With `up` set, the
// stripe is R / 2 rows of `src` (gate) then the R / 2 matching rows of `up`.
__global__ __launch_bounds__(256) void tile_kernel(const uint16_t* __restrict__ src, const uint16_t* __restrict__ up,
                                                   int rows, int din, int ld, int ns, int kt, int R,
                                                   uint16_t* __restrict__ dst) {
  const size_t c = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= (size_t)ns * kt * 4 * R) return;
  const int n = (int)(c % R);
  const size_t q = c / R;
  const int kg = (int)(q % 4);
  const size_t st = q / 4;
  const int t = (int)(st % kt), s = (int)(st / kt);
  const int k0 = 32 * t + 8 * kg;
  const uint16_t* base = src;
  int row = R * s + n;
  if (up) {
    const int U = R / 2;
    row = U * s + (n % U);
    base = n < U ? src : up;
  }
  v4u v = {0u, 0u, 0u, 0u};
  if (row < rows && k0 < din) v = *reinterpret_cast<const v4u*>(base + (size_t)row * ld + k0);
  reinterpret_cast<v4u*>(dst)[c] = v;
}

}  // namespace

void mfma_split_need(int mode, int ns, int kt, int rh, int batch, size_t* kpart_floats, size_t* tickets) {
  const SplitGeom g = split_geom(static_cast<MMode>(mode), ns, kt, rh, nbt_of(batch));
  const size_t ny = (batch + kGroupSeq - 1) / kGroupSeq;
  const size_t nout = (size_t)nbt_of(batch) * kSeqTile * 16;
  *kpart_floats = g.ks > 1 ? ny * g.ngr * g.ks * g.nstr_max * nout : 0;
  *tickets = g.ks > 1 ? ny * g.ngr : 0;
}

hipError_t launch_mfma_qkv(const MfmaArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mmode<MMode::kQkv>(a, s, ev);
}
hipError_t launch_mfma_oproj(const MfmaArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mmode<MMode::kOproj>(a, s, ev);
}
hipError_t launch_mfma_gate_up(const MfmaArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mmode<MMode::kGateUp>(a, s, ev);
}
hipError_t launch_mfma_down(const MfmaArgs& a, hipStream_t s, KernelEvents ev) {
  return launch_mmode<MMode::kDown>(a, s, ev);
}

hipError_t launch_tile_weights(const uint16_t* src, const uint16_t* up, int rows, int din, int ld, int ns, int kt,
                               int rh, uint16_t* dst, hipStream_t s) {
  const size_t n = (size_t)ns * kt * 4 * rh;
  const unsigned blocks = (unsigned)((n + 255) / 256);
  hipLaunchKernelGGL(tile_kernel, dim3(blocks), dim3(256), 0, s, src, up, rows, din, ld, ns, kt, rh, dst);
  return hipGetLastError();
}

}  // namespace fasttps
