// The split-KV decode attention of one (split, KV head, sequence) as a
// device-side body, shared by the attention kernel (attention.hip) and the
// fused layer kernel (fused_layer.hip). See attention.hip for the method.
//
// The body runs on 256 threads (a block, or a quarter of the fused kernel's
// block) in three steps:
//   load_prologue()  q, k, v of the item and the RoPE row
//   prime()          the ring's first K/V tiles (they do not depend on q, so
//                    a fused kernel issues them before it waits for the QKV
//                    phase)
//   run()            RoPE, the append, the streaming loop and the split's
//                    (m, l, o)
// The q|k|v reads and the (m, l, o) writes go through an IO policy (plain
// global memory, or agent-coherent accesses in the fused kernel).
#pragma once

#include <math.h>

#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace fasttps {
namespace attn {


constexpr int kThreads = 256;
constexpr int kTile = 64;         // positions per tile (4 lanes each)

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

using fasttps::merge_factor;

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
// `last`, a position of this split), quarter `seg` of the row. Plain loads:
// the three chunks of a lane's quarter row are three load instructions, and
// each of them touches every 128-byte line of the 16 rows the wave reads, so
// the lines must stay in L2 between them; with the non-temporal policy of the
// weight streams the Phi-3 attention at KV 4096 took 15.0 instead of 11.4 us
// on MI355X.
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

// The contiguous variant (bf16 cache): a wave's 16 positions of a tile are
// 16 consecutive rows, one contiguous span of 16 RC16 16-byte chunks; lane l
// loads chunks l, l + 64, ... of it (each load instruction one contiguous
// kilobyte, whole 128-byte lines), with the non-temporal policy of the
// weight streams; rows past `last` are clamped to it. The chunks reach the
// lanes that compute with them through the wave's LDS exchange area.
template <int RC16, int NC>
__device__ __forceinline__ void tile_load_contig(v4u (&k)[NC], v4u (&v)[NC], const v4u* __restrict__ Kc,
                                                 const v4u* __restrict__ Vc, int t0, int last, int wave, int lane) {
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int q = lane + kWave * c;
    const size_t at = (size_t)min(t0 + 16 * wave + q / RC16, last) * RC16 + q % RC16;
    k[c] = ld_stream(Kc + at);
    v[c] = ld_stream(Vc + at);
  }
}

// Plain global-memory IO of the attention kernel. rec() is where the split's
// record (m, l, -, -, o) of query head `head` of sequence b goes.
struct GlobalIO {
  __device__ __forceinline__ float qkv(const AttnArgs& a, size_t i) const { return a.qkv[i]; }
  __device__ __forceinline__ void part(float* p, float v) const { *p = v; }
  __device__ __forceinline__ float* rec(const AttnArgs& a, int b, int head, int s, int D) const {
    return a.part + (((size_t)b * a.n_heads + head) * a.nsplit_cap + s) * (D + kPartLead);
  }
};

// PBF16: the softmax weights enter PV rounded to bf16, as FlashAttention's
// bf16 P does (the row sum l keeps the fp32 weights); the accuracy study
// compares this with the fp32 path. The step itself uses PBF16 = false.
// KVF: the cache's element format; kscale and vscale are the KV head's scales
// of an 8-bit cache (unused for bf16). live = false runs the item's barriers
// and nothing else (no positions, no stores), for a quarter of a fused block
// without an item.
// XCH: the contiguous loads and the LDS exchange (bf16 caches; xk, xv each
// hold kThreads / kWave spans of 16 RC rows, one per wave); otherwise each
// lane loads its quarter rows itself with plain loads.
template <int D, int G, int NRING, bool PBF16, int KVF, class IO, bool XCH = false>
struct AttnBody {
  using R = LaneRow<D, KVF>;
  using Chunk = typename R::Chunk;
  static constexpr int SEG = D / 4;   // elements of a position row per lane
  static constexpr int NC = R::NC;    // chunks per lane (K and V each)
  static constexpr int RC = D * kv_bytes<KVF>() / 16;  // 16-byte chunks per row (the append)
  static constexpr int HALF = D / 2;
  static constexpr int SPAN = 16 * RC;  // chunks of a wave's 16 rows (XCH)
  static_assert(SEG == NC * R::EPC, "a lane's quarter row must be whole chunks");
  static_assert(G * HALF <= kThreads && D <= kThreads, "one prologue element per thread");
  static_assert(!XCH || (KVF == kKvBf16 && SPAN == kWave * NC), "the exchange covers a wave's rows in NC loads");
  using Smem = AttnSmem<D, G, KVF>;

  const AttnArgs& a;
  IO io;
  Smem& sm;
  v4u* xk;  // XCH: this wave's exchange spans (LDS)
  v4u* xv;
  int tid, s, g, b, P, start, stride, end, last, j, seg, pj, ph;
  bool own_new, live;
  size_t head_off;
  const Chunk* Kc;
  const Chunk* Vc;
  double c_j, s_j;
  float q0, q1, k0, k1, v0;
  Chunk kr[NRING][NC], vr[NRING][NC];

  // nsplit_: the splits the tiles are dealt to (0: a.nsplit)
  __device__ __forceinline__ AttnBody(const AttnArgs& a_, IO io_, Smem& sm_, int tid_, int s_, int g_, int b_,
                                      bool live_, v4u* xk_ = nullptr, v4u* xv_ = nullptr, int nsplit_ = 0)
      : a(a_), io(io_), sm(sm_), tid(tid_), s(s_), g(g_), b(b_), live(live_) {
    const int nsp = nsplit_ ? nsplit_ : a.nsplit;
    xk = xk_ + (tid_ / kWave) * SPAN;
    xv = xv_ + (tid_ / kWave) * SPAN;
    P = a.pos.p[b];
    // tiles s, s + nsplit, ... of the sequence's cached entries [0, P); the
    // new entry P is added from LDS by the split whose tile index holds it
    start = s * kTile;
    stride = nsp * kTile;
    end = live ? P : start;
    last = max(P - 1, 0);  // loads past the end read this cached row (masked); slot P is never read
                           // unless P = 0, where the clamped prime loads read slot 0 and discard it
    head_off = ((size_t)b * a.n_kv_heads + g) * (size_t)a.max_seq * D * kv_bytes<KVF>();  // bytes
    Kc = reinterpret_cast<const Chunk*>(static_cast<const uint8_t*>(a.k_cache) + head_off);
    Vc = reinterpret_cast<const Chunk*>(static_cast<const uint8_t*>(a.v_cache) + head_off);
    j = tid >> 2;
    seg = tid & 3;
    own_new = live && (P / kTile) % nsp == s;  // the split whose tile holds slot P
    pj = tid % HALF;
    ph = min(tid / HALF, G - 1);
  }

  // ---- prologue operands (every thread loads; clamped) ---------------------
  __device__ __forceinline__ void load_prologue() {
    const int H = a.n_heads, Hkv = a.n_kv_heads;
    const size_t rowlen = (size_t)(H + 2 * Hkv) * D;
    const size_t qkv = (size_t)b * rowlen;
    const size_t qg = qkv + (size_t)g * G * D;
    const size_t kg = qkv + (size_t)H * D + (size_t)g * D;
    const size_t vg = qkv + (size_t)(H + Hkv) * D + (size_t)g * D;
    const double* cs = a.rope_cos + (size_t)P * HALF;
    const double* sn = a.rope_sin + (size_t)P * HALF;
    c_j = cs[pj];
    s_j = sn[pj];
    q0 = io.qkv(a, qg + ph * D + pj);
    q1 = io.qkv(a, qg + ph * D + pj + HALF);
    k0 = io.qkv(a, kg + pj);
    k1 = io.qkv(a, kg + pj + HALF);
    v0 = io.qkv(a, vg + tid % D);
  }

  // ---- the ring's first NRING tiles ----------------------------------------
  __device__ __forceinline__ void prime() {
#pragma unroll
    for (int r = 0; r < NRING; ++r) refill(r, start + r * stride);
  }

  // ring slot r <- the tile at t0
  __device__ __forceinline__ void refill(int r, int t0) {
    if constexpr (XCH)
      tile_load_contig<RC, NC>(kr[r], vr[r], Kc, Vc, t0, last, tid / kWave, tid % kWave);
    else
      tile_load<R::ROW_CHUNKS>(kr[r], vr[r], Kc, Vc, t0, last, j, seg);
  }

  // this lane's quarter rows of ring slot r: the slot itself, or (XCH) its
  // chunks through the wave's exchange spans (wave-private, so no block
  // barrier: a wave's LDS accesses take effect in program order). A lane
  // reads what other lanes wrote, which no per-lane dependence expresses, so
  // wavefront-scope fences keep every write before the reads and the reads
  // before the next slot's writes (without them the compiler may interleave
  // them, and the exchange reads stale chunks)
  __device__ __forceinline__ void lane_rows(int r, Chunk (&kq)[NC], Chunk (&vq)[NC]) {
    if constexpr (XCH) {
      const int lane = tid % kWave;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        xk[lane + kWave * c] = kr[r][c];
        xv[lane + kWave * c] = vr[r][c];
      }
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      const int at = (lane >> 2) * RC + (lane & 3) * NC;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        kq[c] = xk[at + c];
        vq[c] = xv[at + c];
      }
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    } else {
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        kq[c] = kr[r][c];
        vq[c] = vr[r][c];
      }
    }
  }

  __device__ __forceinline__ void run(float kscale, float vscale) {
    // ---- prologue: RoPE in double, rounding of the new K/V ------------------
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
      uint8_t* dst = static_cast<uint8_t*>(isv ? a.v_cache : a.k_cache) + head_off + (size_t)P * D * kv_bytes<KVF>();
      reinterpret_cast<v4u*>(dst)[c] = val;
    }
    // this lane's quarter of the query heads: registers for one head, LDS
    // (read as a broadcast) for a group
    float qr[G == 1 ? SEG : 1];
    if (G == 1) {
#pragma unroll
      for (int e = 0; e < SEG; ++e) qr[e] = sm.q[0][seg * SEG + e];
    }

    // ---- main loop over the split's tiles: its cached entries below P -----
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
    // ring slot r holds tile tt: its update, and (REFILL) the slot's refill
    // with the tile NRING further on (clamped past the end); the barrier keeps
    // the refill after the unpack, so the new tile lands in the registers the
    // old one leaves (no copies, no early waits)
    auto slot = [&](int r, int tt, auto refill_tag) {
      float kf[SEG], vf[SEG];
      {
        Chunk kq[NC], vq[NC];
        lane_rows(r, kq, vq);
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          decode_chunk<KVF>(kq[c], kf + R::EPC * c);
          decode_chunk<KVF>(vq[c], vf + R::EPC * c);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (decltype(refill_tag)::value) refill(r, tt + NRING * stride);
      update(kf, vf, tt + j < end);
    };
    // the last round refills nothing: its refills would be loads past the
    // split that the merge below waits for (it reuses their registers)
    int t0 = start;
    for (; t0 + NRING * stride < end; t0 += NRING * stride) {
#pragma unroll
      for (int r = 0; r < NRING; ++r) slot(r, t0 + r * stride, BoolTag<true>{});
    }
    if (t0 < end) {
#pragma unroll
      for (int r = 0; r < NRING; ++r) slot(r, t0 + r * stride, BoolTag<false>{});
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

    // test hook: q and k after RoPE (fp32), written after the stream by the
    // split that owns the new entry
    if (a.dbg_qk && own_new) {
      const int H = a.n_heads, Hkv = a.n_kv_heads;
      float* dq = a.dbg_qk + (size_t)b * (H + Hkv) * D;
      for (int i = tid; i < G * D; i += kThreads) dq[(size_t)g * G * D + i] = sm.q[i / D][i % D];
      if (tid < HALF) {
        // k and its cos/sin row again from memory (not held across the loop)
        const size_t kg = (size_t)b * (H + 2 * Hkv) * D + (size_t)H * D + (size_t)g * D;
        const double kk0 = a.qkv[kg + pj], kk1 = a.qkv[kg + pj + HALF];
        const double c = a.rope_cos[(size_t)P * HALF + pj], sn = a.rope_sin[(size_t)P * HALF + pj];
        float* dk = dq + (size_t)H * D + (size_t)g * D;
        dk[pj] = (float)(kk0 * c - kk1 * sn);
        dk[pj + HALF] = (float)(kk1 * c + kk0 * sn);
      }
    }

    // ---- merge: the 4 positions of each 16-lane row (DPP), then the rows --
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

    if (!live) return;
    // element i of the G heads' o by the lane pair (2i', 2i' + 1) of the
    // block's threads, each lane over half of the 16 rows; the pair adds its
    // halves with one lane swap (every thread takes part: the merge is the
    // block's last step and nothing else hides its latency)
    constexpr int kHalfRows = kRows / 2;
    for (int i0 = 0; i0 < G * D; i0 += kThreads / 2) {
      const int i = min(i0 + tid / 2, G * D - 1), hr = tid & 1;
      const int h = i / D, e = i % D;
      float M = sm.rm[h][0];
#pragma unroll
      for (int r = 1; r < kRows; ++r) M = fmaxf(M, sm.rm[h][r]);
      float L = 0.f, O = 0.f;
#pragma unroll
      for (int q = 0; q < kHalfRows; ++q) {
        const int r = hr * kHalfRows + q;
        const float f = merge_factor(sm.rm[h][r], M);
        L = fmaf(sm.rl[h][r], f, L);
        O = fmaf(sm.red[h][r][e], f, O);
      }
      L += dpp_mov<kDppQuadXor1>(L);
      O += dpp_mov<kDppQuadXor1>(O);
      if (hr == 0 && i0 + tid / 2 < G * D) {
        float* pr = io.rec(a, b, g * G + h, s, D);
        io.part(pr + kPartLead + e, KVF == kKvBf16 ? O : O * vscale);  // an 8-bit cache's V scale
        if (e == 0) {
          io.part(pr, M);
          io.part(pr + 1, L);
        }
      }
    }
  }
};

}  // namespace attn
}  // namespace fasttps
