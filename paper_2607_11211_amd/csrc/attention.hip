// Decode attention with joint RoPE, in-place cache append and split-KV (gfx950).
//
// The paper's TPSFLAT (Alg. 3, Section 3.1.2) runs RoPE, the K append, QK^T,
// softmax and PV for one head inside one core's L1. One head's work is far
// too small for a 256-CU chip, so here the softmax-independent axis the paper
// uses (heads) is combined with a split of the cached positions:
//   grid = (split, kv head g, sequence b), the sequences in order of
//   decreasing length (the blocks go out in grid order, so the shortest
//   blocks fill the end of the kernel); of the tiles of 64 positions of
//   one (b, g), split s of S takes tiles s, s + S, s + 2S, ... for all
//   G = H/H_kv query heads of that KV head, so each K/V byte is read from HBM
//   once (grouped-query attention). The splits of a head are interleaved
//   rather than contiguous ranges so that at any moment the blocks of a head
//   read one compact window of the cache, as the GEMVs deal their rows
//   (contiguous ranges left some split lengths of the batched and ragged
//   workloads several percent slower on MI355X).
// Per block (256 threads, tiles of 64 positions):
//   * four lanes share a position, each owning a quarter of d: a lane loads
//     exactly the K and V chunks it computes with (the four lanes of a
//     position read one contiguous row), straight into registers, with a
//     ring of NRING tiles in flight. No tile passes through LDS and the loop
//     has no barrier;
//   * the prologue's few loads go out first, then the ring: a wave's loads
//     return in the order they were issued. Every load is issued
//     unconditionally (rows past the sequence are clamped to its last entry
//     and masked),
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
// log-sum-exp identity (one wave per (b, head) up to 32 splits, a block
// beyond). A merge inside the split launch (each block stores its state
// with coherent stores, waits for them and takes a ticket of its (sequence,
// KV head); the last one merges) was measured slower on MI355X: the store
// acknowledgements and the ticket's round trip under full HBM load hold
// every block longer than the merge launch costs (Phi-3 layer at KV 4096:
// attention 12.0 -> 16.0 us against a 4.4 us merge kernel, 59.9 -> 61.7 us
// per layer; 16-sequence ragged batch: attention 75.9 -> 87.2 us).
#include "attn_body.h"

namespace fasttps {

namespace {

using attn::kThreads;
using attn::merge_factor;

constexpr int kMaxSplits = 256;   // splits per (sequence, kv head); one combine thread each
// bf16 caches: whole-line non-temporal loads and the LDS exchange (AttnBody
// XCH) for one or two query heads per KV head and splits of at least
// kXchMinTiles tiles. Measured on MI355X (per layer step, HIP graph): the
// 16-sequence ragged Phi-3 batch (splits of 9 tiles) attention 88.3 -> 77.0
// us; Phi-3 at KV 4096 (4 tiles) 11.45 -> 11.42; at KV 1024 (1 tile) 5.65 ->
// 7.28; the GQA layer (groups of four, one tile in flight per lane at 256
// VGPRs) 105.8 -> 124.3.
constexpr int kXchMinTiles = 8;

// one (split, KV head, sequence) per block
template <int D, int G, int NRING, bool PBF16, int KVF, bool XCH>
__device__ __forceinline__ void attn_split_body(const AttnArgs& a, float kscale, float vscale) {
  using Body = attn::AttnBody<D, G, NRING, PBF16, KVF, attn::GlobalIO, XCH>;
  __shared__ attn::AttnSmem<D, G, KVF> sm;
  __shared__ v4u xch[XCH ? 2 * (kThreads / kWave) * Body::SPAN : 1];  // K spans, then V spans
  Body body(a, attn::GlobalIO{}, sm, threadIdx.x, blockIdx.x, blockIdx.y, a.order.p[blockIdx.z], true, xch,
            xch + (kThreads / kWave) * Body::SPAN);
  body.load_prologue();
  __builtin_amdgcn_sched_barrier(0);  // keep the prologue loads ahead of the tiles
  body.prime();
  body.run(kscale, vscale);
}

// At least two waves per SIMD: the groups of four at d = 128 (one tile in
// flight per lane, o of four heads in registers) then fit 256 registers
// without spilling, so two blocks share a CU instead of one.
template <int D, int G, int NRING, bool PBF16, bool XCH>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 8))) void attn_split_kernel(AttnArgs a) {
  attn_split_body<D, G, NRING, PBF16, kKvBf16, XCH>(a, 1.f, 1.f);
}

// 8-bit cache: the KV head's two scales come from the argument block; tiles
// in flight as for a bf16 cache
template <int D, int G, int KVF>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 8))) void attn_split_kv8_kernel(
    AttnArgs a, KvScales sc) {
  attn_split_body<D, G, (G <= 2 ? 2 : 1), false, KVF, false>(a, sc.k[blockIdx.y], sc.v[blockIdx.y]);
}

// o[b, h] = sum_s e^{m_s - M} o_s / sum_s e^{m_s - M} l_s,  M = max_s m_s.
// One block of 1024 threads per (head, sequence), for more than 32 splits.
// Every load is issued up front (the o rows do not depend on M), so the
// kernel costs one round trip: thread s reads split s's (m, l); thread
// (group, e) reads o_s[e] of the splits s = group, group + NG, ... (NG =
// 1024 / D groups, at most 32 splits each). A 256-thread version that looped
// over the splits past its registers, one dependent load at a time, took
// 22 us for 128 splits at d = 128.
constexpr int kCombineThreads = 1024;
constexpr int kCombineRegs = 32;  // splits per thread held in registers
static_assert(kCombineThreads / 128 * kCombineRegs >= kMaxSplits, "one round of loads covers every split");

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
  const float* ph = part + ((size_t)b * n_heads + h) * nsplit_cap * (D + kPartLead);
  const int grp = tid / D, e = tid % D;
  float ov[kCombineRegs];
#pragma unroll
  for (int k = 0; k < kCombineRegs; ++k) {
    const int q = grp + NG * k;
    ov[k] = (grp < NG && q < nsplit) ? ph[(size_t)q * (D + kPartLead) + kPartLead + e] : 0.f;
  }
  const float ms = tid < nsplit ? ph[(size_t)tid * (D + kPartLead)] : -INFINITY;
  const float ls = tid < nsplit ? ph[(size_t)tid * (D + kPartLead) + 1] : 0.f;
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

// The same merge by one wave per (head, sequence), for up to NS = 16 or 32
// splits: lane s reads split s's (m, l); the o values of NS splits are loaded
// up front (one round trip) and merged with each split's factor read from
// lane s. No block barrier: on the batch-1 Phi-3 layer this saved ~0.5 us per
// step against a 256-thread block version, and loading 16 splits instead of
// 32 for its 16 splits another ~0.3 us. Past 32 splits it would need a second
// round trip, which made it slower than the block kernel (7.2 us for 64
// splits at d = 128, against 4.9 us for 128 splits in the block kernel).
constexpr int kWaveCombineSplits = 32;
template <int D, int NS>
__global__ __launch_bounds__(kWave) void attn_combine_wave_kernel(const float* __restrict__ part, int nsplit,
                                                                 int nsplit_cap, int n_heads, float* __restrict__ o,
                                                                 uint16_t* __restrict__ o_operand, int o_nbtc) {
  constexpr int EPL = (D + kWave - 1) / kWave;  // o elements per lane
  const int lane = threadIdx.x;
  const int h = blockIdx.x, b = blockIdx.y;
  const float* ph = part + ((size_t)b * n_heads + h) * nsplit_cap * (D + kPartLead);
  const int sl = min(lane, nsplit - 1);
  const float ms = lane < nsplit ? ph[(size_t)sl * (D + kPartLead)] : -INFINITY;
  const float ls = lane < nsplit ? ph[(size_t)sl * (D + kPartLead) + 1] : 0.f;
  float ov[NS][EPL];
#pragma unroll
  for (int j = 0; j < NS; ++j)
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      ov[j][i] = ph[(size_t)min(j, nsplit - 1) * (D + kPartLead) + kPartLead + min(lane + kWave * i, D - 1)];
  const float M = wave_max(ms);
  const float f = merge_factor(ms, M);  // zero for lanes past the splits
  const float L = wave_sum(ls * f);
  float acc[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) acc[i] = 0.f;
#pragma unroll
  for (int j = 0; j < NS; ++j) {
    // lanes past the splits hold f = 0
    const float fj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), j));
#pragma unroll
    for (int i = 0; i < EPL; ++i) acc[i] = fmaf(ov[j][i], fj, acc[i]);
  }
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane + kWave * i;
    if (e < D) {
      const float v = acc[i] / L;
      o[((size_t)b * n_heads + h) * D + e] = v;
      if (o_operand) {
        // the MFMA O projection's operand, as in attn_combine_kernel
        const int k = h * D + e;
        const uint16_t hi = f32_to_bf16(v);
        const uint16_t lo = f32_to_bf16(v - bf16_to_f32(hi));
        const size_t base = (((size_t)(k >> 5) * o_nbtc + b / 8) * kWave + 2 * (b % 8) + 16 * ((k >> 3) & 3)) * 8 +
                            (k & 7);
        o_operand[base] = hi;
        o_operand[base + 8] = lo;
      }
    }
  }
}

template <int D, int G>
hipError_t launch_dg(const AttnArgs& a, hipStream_t s, KernelEvents ev) {
  // tiles in flight per lane: a tile is D / 8 registers of K and V; the
  // query quarter and the softmax state take (D / 4 + 2) G more. Two for one
  // or two query heads (103-226 VGPRs at d = 64-128: at least the two blocks
  // per CU the split targets), one for groups of four (up to 256 VGPRs).
  // A group of four as two blocks of two heads each (two tiles in flight,
  // the pair reading the same K/V tiles at about the same time) was measured
  // slower on MI355X: GQA layer at 4 x 32768, attention 96.2 -> 116.8 us
  // (plain loads) and 124.3 us (whole-line non-temporal loads); the pair's
  // second reads do not come from cache often enough.
  constexpr int NRING = G <= 2 ? 2 : 1;
  dim3 grid(a.nsplit, a.n_kv_heads, a.batch);
  int maxp = 0;
  for (int b = 0; b < a.batch; ++b) maxp = a.pos.p[b] > maxp ? a.pos.p[b] : maxp;
  const int tiles = (maxp + attn::kTile - 1) / attn::kTile;
  if constexpr (G <= 2) {
    if ((tiles + a.nsplit - 1) / a.nsplit >= kXchMinTiles)
      return a.p_bf16 ? ext_launch(attn_split_kernel<D, G, NRING, true, true>, grid, dim3(kThreads), 0, s, ev, a)
                      : ext_launch(attn_split_kernel<D, G, NRING, false, true>, grid, dim3(kThreads), 0, s, ev, a);
  }
  return a.p_bf16 ? ext_launch(attn_split_kernel<D, G, NRING, true, false>, grid, dim3(kThreads), 0, s, ev, a)
                  : ext_launch(attn_split_kernel<D, G, NRING, false, false>, grid, dim3(kThreads), 0, s, ev, a);
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
  if (a.nsplit <= kWaveCombineSplits / 2)
    return ext_launch(attn_combine_wave_kernel<D, kWaveCombineSplits / 2>, grid, dim3(kWave), 0, s, ev,
                      (const float*)a.part, a.nsplit, a.nsplit_cap, a.n_heads, a.o, a.o_operand, a.o_nbtc);
  if (a.nsplit <= kWaveCombineSplits)
    return ext_launch(attn_combine_wave_kernel<D, kWaveCombineSplits>, grid, dim3(kWave), 0, s, ev,
                      (const float*)a.part, a.nsplit, a.nsplit_cap, a.n_heads, a.o, a.o_operand, a.o_nbtc);
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
