// Decode attention with joint RoPE, in-place cache append and split-KV (gfx950).
//
// The paper's TPSFLAT (Alg. 3, Section 3.1.2) runs RoPE, the K append, QK^T,
// softmax and PV for one head inside one core's L1. One head's work is far
// too small for a 256-CU chip, so here the softmax-independent axis the paper
// uses (heads) is combined with a split of the cached positions:
//   grid = (split, kv head g, sequence b); a block covers positions
//   [s*L, s*L + L) of one (b, g) for all G = H/H_kv query heads of that KV
//   head, so each K/V byte is read from HBM once (grouped-query attention).
// Per block (256 threads, tiles of 64 positions):
//   * four lanes share a position, each owning a quarter of d: a lane loads
//     exactly the K and V chunks it computes with (the four lanes of a
//     position read one contiguous row), straight into registers, with a
//     ring of NRING tiles in flight. No tile passes through LDS and the loop
//     has no barrier;
//   * the prologue's few loads go out first, then the ring: a wave's loads
//     return in the order they were issued. Every load is issued
//     unconditionally (rows past the split are clamped into it and masked),
//     so the compiler waits for exactly the tile it needs;
//   * prologue: RoPE on the G query heads and on k, with shared cos/sin rows
//     in double precision (Alg. 3 joint RoPE; Eq. 22); the block that owns the
//     new position N_p rounds k and v to bf16 and writes them to slot N_p
//     (GKVC, Eq. 1). The lanes of position N_p take the rounded values from
//     LDS: slot N_p is never read back from memory and no other block
//     touches it;
//   * QK^T partials are finished with two in-quad DPP moves, and each lane
//     keeps an online-softmax state (m, l, o-quarter) per query head;
//   * the block merges its lanes' states (DPP within each 16-lane row, then
//     the 16 rows through LDS) and writes (m, l, o) for its split.
// The same kernel also serves an 8-bit cache (FP8 E4M3 or INT8 codes, one
// scale per KV head for K and for V): a lane then loads d/4 bytes of a row,
// decodes them with the hardware FP8 converts (or sign-extending byte
// extracts), and the scales are folded into the softmax scale (K) and the
// split's output (V); the new entry is rounded onto the 8-bit grid once, in
// double precision, before it is stored and used.
// A second small kernel combines the splits of each (b, head) with the
// log-sum-exp identity. (Cross-block tickets are avoided on purpose: on this
// chip an agent-scope fence per block costs far more than a kernel boundary.)
#include "common.h"
#include "kernels.h"

#include <math.h>

#include <type_traits>

namespace fasttps {

namespace {

constexpr int kThreads = 256;
constexpr int kTile = 64;         // positions per tile (4 lanes each)
constexpr int kMaxSplits = 256;   // splits per (sequence, kv head); one combine thread each

constexpr int kRows = kThreads / 16;  // 16-lane DPP rows per block (4 positions each)
// Online softmax with a lazily moved reference (natural-log units): a lane's
// weights e^(s - m) stay below e^8 ~ 3e3, so l and o stay far from fp32 range
// limits over any split, and (m, l, o) of different lanes and splits combine
// exactly as before (any reference m works in the log-sum-exp merge).
constexpr float kLazyRescale = 8.0f;

typedef unsigned int v2u __attribute__((ext_vector_type(2)));
typedef float v2f __attribute__((ext_vector_type(2)));

// bytes per cache element
template <int KVF>
constexpr int kv_bytes() { return KVF == kKvBf16 ? 2 : 1; }

// A lane's quarter of one cache row: D / 4 elements in NC chunks of CB bytes
// (16-byte chunks where the quarter allows, else 8-byte ones: a d = 96 row of
// 8-bit codes gives 24 bytes per lane).
template <int D, int KVF>
struct LaneRow {
  static constexpr int BYTES = D / 4 * kv_bytes<KVF>();
  static constexpr int CB = BYTES % 16 == 0 ? 16 : 8;
  static constexpr int NC = BYTES / CB;
  static constexpr int EPC = CB / kv_bytes<KVF>();        // elements per chunk
  static constexpr int ROW_CHUNKS = D * kv_bytes<KVF>() / CB;
  typedef typename std::conditional<CB == 16, v4u, v2u>::type Chunk;
};

template <int D, int G, int KVF>
struct alignas(16) AttnSmem {
  float q[G][D];
  alignas(16) uint8_t knew[D * kv_bytes<KVF>()];  // the new entry as stored
  alignas(16) uint8_t vnew[D * kv_bytes<KVF>()];
  float red[G][kRows][D];  // the rows' o sums
  float rm[G][kRows];      // the rows' running max and sum
  float rl[G][kRows];
};

__device__ __forceinline__ float merge_factor(float m, float M) {
  return (m == -INFINITY) ? 0.f : __expf(m - M);
}

// four codes of one 32-bit word, element 4i + k in byte k
template <int KVF>
__device__ __forceinline__ void decode_word(uint32_t w, float* f) {
  if constexpr (KVF == kKvFp8) {
    const v2f lo = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, false);
    const v2f hi = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, true);
    f[0] = lo.x; f[1] = lo.y; f[2] = hi.x; f[3] = hi.y;
  } else {
    f[0] = (float)((int)(w << 24) >> 24);
    f[1] = (float)((int)(w << 16) >> 24);
    f[2] = (float)((int)(w << 8) >> 24);
    f[3] = (float)((int)w >> 24);
  }
}

// the EPC elements of one chunk as floats (unscaled codes for 8-bit caches)
template <int KVF>
__device__ __forceinline__ void decode_chunk(const v4u c, float* f) {
  if constexpr (KVF == kKvBf16) {
    unpack8(c, f);
  } else {
    decode_word<KVF>(c.x, f); decode_word<KVF>(c.y, f + 4);
    decode_word<KVF>(c.z, f + 8); decode_word<KVF>(c.w, f + 12);
  }
}
template <int KVF>
__device__ __forceinline__ void decode_chunk(const v2u c, float* f) {
  static_assert(KVF != kKvBf16, "bf16 rows use 16-byte chunks");
  decode_word<KVF>(c.x, f); decode_word<KVF>(c.y, f + 4);
}

// The E4M3 code (OCP: bias 7, subnormals, largest finite 448) of a double:
// nearest value, ties to the even code, magnitudes from 448 up saturating;
// the sign bit is the sign of x. The quantum is 2^(e - 3) in the binade
// [2^e, 2^(e+1)), e >= -6, and 2^-9 below (subnormals).
__device__ __forceinline__ uint8_t f64_to_e4m3(double x) {
  const uint32_t sign = signbit(x) ? 0x80u : 0u;
  const double ax = fabs(x);
  if (!(ax < 448.0)) return (uint8_t)(sign | 0x7Eu);
  if (ax == 0.0) return (uint8_t)sign;
  const int lead = ilogb(ax);                   // ax in [2^lead, 2^(lead+1))
  const int qe = (lead < -6 ? -6 : lead) - 3;
  const int q = (int)rint(ldexp(ax, -qe));      // nearest even; 0 .. 16
  if (lead < -6) return (uint8_t)(sign | (uint32_t)q);  // subnormal, or 8 = 2^-6
  const int e = q == 16 ? lead + 1 : lead;
  const int m = q == 16 ? 0 : q - 8;
  return (uint8_t)(sign | (uint32_t)((e + 7) << 3) | (uint32_t)m);
}

// The INT8 code of a double: nearest integer (ties to even), clamped to
// [-127, 127], as its two's-complement byte.
__device__ __forceinline__ uint8_t f64_to_int8(double x) {
  const double r = fmin(fmax(rint(x), -127.0), 127.0);
  return (uint8_t)(int8_t)(int)r;
}

// element e of the new entry, stored into the LDS row: bf16 of x, or the
// 8-bit code of x / s
template <int KVF>
__device__ __forceinline__ void store_new(uint8_t* row, int e, double x, double s) {
  if constexpr (KVF == kKvBf16) {
    reinterpret_cast<uint16_t*>(row)[e] = f64_to_bf16(x);
  } else if constexpr (KVF == kKvFp8) {
    row[e] = f64_to_e4m3(x / s);
  } else {
    row[e] = f64_to_int8(x / s);
  }
}

// This lane's K and V chunks of the tile at t0: position t0 + j (clamped to
// `last`, a position of this split), quarter `seg` of the row.
template <int ROW_CHUNKS, int NC, typename Chunk>
__device__ __forceinline__ void tile_load(Chunk (&k)[NC], Chunk (&v)[NC], const Chunk* __restrict__ Kc,
                                          const Chunk* __restrict__ Vc, int t0, int last, int j, int seg) {
  const size_t base = (size_t)min(t0 + j, last) * ROW_CHUNKS + seg * NC;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    k[c] = Kc[base + c];
    v[c] = Vc[base + c];
  }
}

// PBF16: the softmax weights enter PV rounded to bf16, as FlashAttention's
// bf16 P does (the row sum l keeps the fp32 weights); the accuracy study
// compares this with the fp32 path. The step itself uses PBF16 = false.
// KVF: the cache's element format; kscale and vscale are the KV head's scales
// of an 8-bit cache (unused for bf16).
template <int D, int G, int NRING, bool PBF16, int KVF>
__device__ __forceinline__ void attn_split_body(const AttnArgs& a, float kscale, float vscale) {
  using R = LaneRow<D, KVF>;
  using Chunk = typename R::Chunk;
  constexpr int SEG = D / 4;   // elements of a position row per lane
  constexpr int NC = R::NC;    // chunks per lane (K and V each)
  constexpr int RC = D * kv_bytes<KVF>() / 16;  // 16-byte chunks per row (the append)
  constexpr int HALF = D / 2;
  static_assert(SEG == NC * R::EPC, "a lane's quarter row must be whole chunks");
  __shared__ AttnSmem<D, G, KVF> sm;

  const int tid = threadIdx.x;
  const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int P = a.pos.p[b];
  const int ntot = P + 1;
  const int start = s * a.split_len;
  const int end = min(start + a.split_len, ntot);
  const int last = max(end - 1, start);  // a cache row of this split (start < N_max)
  const int H = a.n_heads, Hkv = a.n_kv_heads;
  const size_t head_off = ((size_t)b * Hkv + g) * (size_t)a.max_seq * D * kv_bytes<KVF>();  // bytes
  const Chunk* Kc = reinterpret_cast<const Chunk*>(static_cast<const uint8_t*>(a.k_cache) + head_off);
  const Chunk* Vc = reinterpret_cast<const Chunk*>(static_cast<const uint8_t*>(a.v_cache) + head_off);
  const int j = tid >> 2, seg = tid & 3;

  // ---- prologue operands first (every thread loads; clamped) ---------------
  const size_t rowlen = (size_t)(H + 2 * Hkv) * D;
  const float* qkv = a.qkv + (size_t)b * rowlen;
  const float* qg = qkv + (size_t)g * G * D;
  const float* kg = qkv + (size_t)H * D + (size_t)g * D;
  const float* vg = qkv + (size_t)(H + Hkv) * D + (size_t)g * D;
  const double* cs = a.rope_cos + (size_t)P * HALF;
  const double* sn = a.rope_sin + (size_t)P * HALF;
  const bool own_new = (start <= P) && (P < end);
  static_assert(G * HALF <= kThreads && D <= kThreads, "one prologue element per thread");
  const int pj = tid % HALF;
  const int ph = min(tid / HALF, G - 1);
  const double c_j = cs[pj], s_j = sn[pj];
  const float q0 = qg[ph * D + pj], q1 = qg[ph * D + pj + HALF];
  const float k0 = kg[pj], k1 = kg[pj + HALF];
  const float v0 = vg[tid % D];
  __builtin_amdgcn_sched_barrier(0);  // keep the prologue loads ahead of the tiles

  // ---- the ring's first NRING tiles ------------------------------------------
  Chunk kr[NRING][NC], vr[NRING][NC];
#pragma unroll
  for (int r = 0; r < NRING; ++r) tile_load<R::ROW_CHUNKS>(kr[r], vr[r], Kc, Vc, start + r * kTile, last, j, seg);

  // ---- prologue: RoPE in double, rounding of the new K/V --------------------
  if (tid < G * HALF) {
    sm.q[ph][pj] = (float)((double)q0 * c_j - (double)q1 * s_j);
    sm.q[ph][pj + HALF] = (float)((double)q1 * c_j + (double)q0 * s_j);
  }
  if (tid < HALF) {
    store_new<KVF>(sm.knew, pj, (double)k0 * c_j - (double)k1 * s_j, (double)kscale);
    store_new<KVF>(sm.knew, pj + HALF, (double)k1 * c_j + (double)k0 * s_j, (double)kscale);
  }
  if (tid < D) {
    if constexpr (KVF == kKvBf16)
      reinterpret_cast<uint16_t*>(sm.vnew)[tid] = f32_to_bf16(v0);
    else
      store_new<KVF>(sm.vnew, tid, (double)v0, (double)vscale);
  }
  __syncthreads();
  // GKVC append (Eq. 1): the one cache write of the step
  if (own_new && tid < 2 * RC) {
    const bool isv = tid >= RC;
    const int c = isv ? tid - RC : tid;
    const v4u val = reinterpret_cast<const v4u*>(isv ? sm.vnew : sm.knew)[c];
    uint8_t* dst = static_cast<uint8_t*>(isv ? a.v_cache : a.k_cache) + head_off +
                   (size_t)P * D * kv_bytes<KVF>();
    reinterpret_cast<v4u*>(dst)[c] = val;
  }
  // this lane's quarter of the query heads: registers for one head, LDS
  // (read as a broadcast) for a group
  float qr[G == 1 ? SEG : 1];
  if (G == 1) {
#pragma unroll
    for (int e = 0; e < SEG; ++e) qr[e] = sm.q[0][seg * SEG + e];
  }

  // ---- main loop over tiles: the cached entries [start, min(end, P)) ------
  float m[G], l[G], o[G][SEG];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY;
    l[h] = 0.f;
#pragma unroll
    for (int e = 0; e < SEG; ++e) o[h][e] = 0.f;
  }
  // an 8-bit cache's K scale folds into the softmax scale
  const float scale = KVF == kKvBf16 ? a.scale : a.scale * kscale;
  const int cend = min(end, P);  // slot P holds the new entry, handled below
  // one step of the online softmax with key kf and value vf
  auto update = [&](const float (&kf)[SEG], const float (&vf)[SEG], bool valid) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float sc = 0.f;
#pragma unroll
      for (int e = 0; e < SEG; ++e) sc = fmaf(G == 1 ? qr[e] : sm.q[h][seg * SEG + e], kf[e], sc);
      sc = quad_sum(sc) * scale;
      if (valid) {
        // the reference m moves only when a score passes it by more than
        // kLazyRescale (then l and o are rescaled once); p = e^(s - m) <=
        // e^kLazyRescale otherwise, and each position costs one FMA per element
        if (sc > m[h] + kLazyRescale) {
          const float cf = merge_factor(m[h], sc);
          l[h] *= cf;
#pragma unroll
          for (int e = 0; e < SEG; ++e) o[h][e] *= cf;
          m[h] = sc;
        }
        const float p = __expf(sc - m[h]);
        l[h] += p;
        const float pv = PBF16 ? bf16_to_f32(f32_to_bf16(p)) : p;
#pragma unroll
        for (int e = 0; e < SEG; ++e) o[h][e] = fmaf(pv, vf[e], o[h][e]);
      }
    }
  };
  for (int t0 = start; t0 < end; t0 += NRING * kTile) {
#pragma unroll
    for (int r = 0; r < NRING; ++r) {
      const int tt = t0 + r * kTile;
      float kf[SEG], vf[SEG];
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        decode_chunk<KVF>(kr[r][c], kf + R::EPC * c);
        decode_chunk<KVF>(vr[r][c], vf + R::EPC * c);
      }
      // refill the slot with the tile NRING further on (clamped past the end);
      // the barrier keeps the refill after the unpack, so the new tile lands
      // in the registers the old one leaves (no copies, no early waits)
      __builtin_amdgcn_sched_barrier(0);
      tile_load<R::ROW_CHUNKS>(kr[r], vr[r], Kc, Vc, tt + NRING * kTile, last, j, seg);
      update(kf, vf, tt + j < cend);
    }
  }
  // the new entry N_p (Eq. 1 slot) from the rounded values in LDS, by the
  // four lanes of position 0
  if (own_new && j == 0) {
    float kf[SEG], vf[SEG];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      decode_chunk<KVF>(reinterpret_cast<const Chunk*>(sm.knew)[seg * NC + c], kf + R::EPC * c);
      decode_chunk<KVF>(reinterpret_cast<const Chunk*>(sm.vnew)[seg * NC + c], vf + R::EPC * c);
    }
    update(kf, vf, true);
  }

  // ---- merge: the 4 positions of each 16-lane row (DPP), then the rows ----
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
    pr[2 + e] = KVF == kKvBf16 ? O : O * vscale;  // an 8-bit cache's V scale
    if (e == 0) {
      pr[0] = M;
      pr[1] = L;
    }
  }
}

template <int D, int G, int NRING, bool PBF16>
__global__ __launch_bounds__(kThreads) void attn_split_kernel(AttnArgs a) {
  attn_split_body<D, G, NRING, PBF16, kKvBf16>(a, 1.f, 1.f);
}

// 8-bit cache: the KV head's two scales come from the argument block
template <int D, int G, int KVF>
__global__ __launch_bounds__(kThreads) void attn_split_kv8_kernel(AttnArgs a, KvScales sc) {
  attn_split_body<D, G, 1, false, KVF>(a, sc.k[blockIdx.y], sc.v[blockIdx.y]);
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
                                                                       float* __restrict__ o,
                                                                       uint16_t* __restrict__ o_operand, int o_nbtc) {
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
    const float ov2 = O / L;
    o[((size_t)b * n_heads + h) * D + tid] = ov2;
    if (o_operand) {
      // the MFMA O projection's operand: hi/lo bf16 split of o at input
      // k = h D + tid, in the lane order of the A operand (row 2 (b % 8) +
      // level, k-group (k / 8) % 4 of k-tile k / 32, batch tile b / 8)
      const int k = h * D + tid;
      const uint16_t hi = f32_to_bf16(ov2);
      const uint16_t lo = f32_to_bf16(ov2 - bf16_to_f32(hi));
      const size_t base = (((size_t)(k >> 5) * o_nbtc + b / 8) * kWave + 2 * (b % 8) + 16 * ((k >> 3) & 3)) * 8 +
                          (k & 7);
      o_operand[base] = hi;
      o_operand[base + 8] = lo;
    }
  }
}

template <int D, int G, int NRING_OVERRIDE = 0>
hipError_t launch_dg(const AttnArgs& a, hipStream_t s, KernelEvents ev) {
  // tiles in flight per lane: a tile is D / 8 registers of K and V; the
  // query quarter and the softmax state take (D / 4 + 2) G more
  constexpr int NRING = NRING_OVERRIDE > 0 ? NRING_OVERRIDE : 1;
  dim3 grid(a.nsplit, a.n_kv_heads, a.batch);
  if (a.p_bf16) return ext_launch(attn_split_kernel<D, G, NRING, true>, grid, dim3(kThreads), 0, s, ev, a);
  return ext_launch(attn_split_kernel<D, G, NRING, false>, grid, dim3(kThreads), 0, s, ev, a);
}

template <int D, int G>
hipError_t launch_kv8_dg(const AttnArgs& a, const KvScales& sc, hipStream_t s, KernelEvents ev) {
  dim3 grid(a.nsplit, a.n_kv_heads, a.batch);
  switch (a.kv_format) {
    case kKvFp8: return ext_launch(attn_split_kv8_kernel<D, G, kKvFp8>, grid, dim3(kThreads), 0, s, ev, a, sc);
    case kKvInt8: return ext_launch(attn_split_kv8_kernel<D, G, kKvInt8>, grid, dim3(kThreads), 0, s, ev, a, sc);
    default: return hipErrorInvalidValue;
  }
}

template <int D>
hipError_t launch_kv8_d(const AttnArgs& a, const KvScales& sc, hipStream_t s, KernelEvents ev) {
  switch (a.n_heads / a.n_kv_heads) {
    case 1: return launch_kv8_dg<D, 1>(a, sc, s, ev);
    case 2: return launch_kv8_dg<D, 2>(a, sc, s, ev);
    case 4: return launch_kv8_dg<D, 4>(a, sc, s, ev);
    default: return hipErrorInvalidValue;
  }
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
                    a.nsplit_cap, a.n_heads, a.o, a.o_operand, a.o_nbtc);
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

hipError_t launch_attention_kv8(const AttnArgs& a, const KvScales& sc, hipStream_t s, KernelEvents ev) {
  if (a.nsplit < 1 || a.nsplit > a.nsplit_cap || a.nsplit > kMaxSplits) return hipErrorInvalidValue;
  if (a.n_kv_heads > kMaxKvHeads) return hipErrorInvalidValue;
  switch (a.head_dim) {
    case 64: return launch_kv8_d<64>(a, sc, s, ev);
    case 96: return launch_kv8_d<96>(a, sc, s, ev);
    case 128: return launch_kv8_d<128>(a, sc, s, ev);
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
