// The whole decode step of one sequence as one persistent kernel (gfx950).
//
// Every launch boundary of the separate kernels costs about 3 us on MI355X
// (the dispatch, the first loads' round trip, the last waves), while the
// weight streams in between run at the chip's read rate. Here one grid of
// 256 blocks x 16 waves (one block per CU) runs the five phases of the step
// in turn: RMSNorm1 + QKV; the attention splits (RoPE, the append, partial
// softmax); the split merge + O projection + residual; RMSNorm2 + gate/up +
// siLu_Mul; the down projection + residual. The paper overlaps weight loads
// with computation inside an operator (Section 3.2 item 3, fine-grain
// pipeline scheduling); here the overlap also crosses the operators: weights
// and cached K/V do not depend on the activation, so a block issues the
// first weight rows (or K/V tiles) of its next phase before it waits for the
// phase that produces that phase's input, and the memory system stays busy
// through the hand-over.
//
// Hand-over between blocks (the L2 caches are per XCD and not coherent):
//   * data another block reads (q|k|v, the split records, h1, the MLP
//     activation) is written with agent-coherent stores and read with
//     agent-coherent loads (sc1), so no L2 write-back or invalidate is needed;
//   * a phase's outputs of a block are written by its wave 0 alone (the GEMV
//     body's segment sums end in wave 0's lanes; the attention's four
//     sub-splits are merged by wave 0), which waits for its stores and then
//     stores the launch's epoch into the block's flag of that phase; the
//     other waves go on to the next phase's prefetch at once;
//   * wave 0 of every block polls the 256 flags of the phase it needs, then
//     a block barrier releases the other waves, whose loads are in flight.
// Every wait is bounded: past kSpinLimit polls the block counts an error
// (read through the debug hook) and goes on, so a grid that could not be
// fully resident ends instead of hanging. The epoch lives in device memory
// and block 0 advances it at its end (every block has read it by then), so
// replays of a captured graph get fresh epochs.
//
// The attention of a block is one (KV head, split) item run as four
// 256-thread sub-bodies on interleaved quarters of the split's tiles (one
// tile in flight per lane, 16 waves per CU), merged in LDS by the
// log-sum-exp identity into the split's record; the O phase merges the
// splits' records of all heads in every block (as oproj_merge_kernel does).
#include "attn_body.h"
#include "gemv_body.h"

#include <algorithm>

namespace fasttps {

namespace {

constexpr int kFThreads = 1024;
constexpr int kSub = kFThreads / attn::kThreads;  // attention sub-bodies per block
constexpr long kSpinLimit = 1L << 18;
constexpr size_t kMaxFusedLds = 160 * 1024;
constexpr int kFusedGrid = 256;                   // one block per CU
constexpr int kFlagsPerLane = kFusedGrid / kWave;  // a wave polls the grid's flags
constexpr int kFusedMaxSplits = 8;                // split records the O phase merges

// 16 bytes at byte offset off of a buffer resource, with the agent-coherent
// policy of ld_c (buffer_load_dwordx4 sc1); the resource is uniform (a
// per-lane base would make the compiler loop over the lanes)
__device__ __forceinline__ float4 ld_c4(__amdgpu_buffer_rsrc_t r, unsigned off) {
  const v4u v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 16);
  return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z), __uint_as_float(v.w));
}

// QKV: x from global memory (written before the launch), outputs coherent
struct QkvIO {
  __device__ __forceinline__ float4 act4(const GemvArgs&, int, int) const { return make_float4(0.f, 0.f, 0.f, 0.f); }
  __device__ __forceinline__ float res(const GemvArgs&, size_t) const { return 0.f; }
  __device__ __forceinline__ void out(const GemvArgs& a, size_t o, float v) const { st_c(a.out + o, v); }
};
// the other projections: the activation from the LDS stage, outputs and
// residuals coherent
struct StageIO {
  const float* stage;
  __device__ __forceinline__ float4 act4(const GemvArgs& a, int b, int i4) const {
    return reinterpret_cast<const float4*>(stage + (size_t)b * a.din)[i4];
  }
  __device__ __forceinline__ float res(const GemvArgs& a, size_t o) const { return ld_c(a.res_f32 + o); }
  __device__ __forceinline__ void out(const GemvArgs& a, size_t o, float v) const { st_c(a.out + o, v); }
};
// attention sub-body of query groups of G heads: q|k|v coherent, its record
// into its LDS slot
template <int G>
struct SubAttnIO {
  float* slot;  // [G][D + kPartLead]
  __device__ __forceinline__ float qkv(const AttnArgs& a, size_t i) const { return ld_c(a.qkv + i); }
  __device__ __forceinline__ void part(float* p, float v) const { *p = v; }
  __device__ __forceinline__ float* rec(const AttnArgs&, int, int head, int, int D) const {
    return slot + (size_t)(head % G) * (D + kPartLead);
  }
};

// wave 0 stored this block's outputs of phase `ph`: it waits for them and
// publishes the block's flag
__device__ __forceinline__ void signal0(const FusedArgs& f, int ph, unsigned epoch) {
  if (threadIdx.x < kWave) {
    wait_vm();
    if (threadIdx.x == 0) st_cu(f.flags + (size_t)ph * gridDim.x + blockIdx.x, epoch);
  }
}

// every block's flag of phase `ph` holds the epoch (wave 0 polls; the block
// barrier then releases the other waves)
__device__ __forceinline__ void wait_phase(const FusedArgs& f, int ph, unsigned epoch) {
  if (threadIdx.x < kWave) {
    const unsigned* fl = f.flags + (size_t)ph * gridDim.x;
    const int lane = threadIdx.x;
    for (long spin = 0;; ++spin) {
      unsigned v[kFlagsPerLane];
#pragma unroll
      for (int k = 0; k < kFlagsPerLane; ++k) v[k] = ld_cu(fl + min(lane + k * kWave, (int)gridDim.x - 1));
      bool ok = true;
#pragma unroll
      for (int k = 0; k < kFlagsPerLane; ++k) ok &= v[k] == epoch;
      if (__all(ok)) break;
      if (spin >= kSpinLimit) {
        if (lane == 0) atomicAdd(f.err, 1);
        break;
      }
    }
  }
  __syncthreads();
}

// the n floats of src into the LDS stage (coherent loads)
__device__ __forceinline__ void stage_in(float* stage, const float* src, int n) {
  for (int i = threadIdx.x; i < n; i += kFThreads) stage[i] = ld_c(src + i);
  __syncthreads();
}

// The step's phases. Q*, O*, GU*, DN*: the launch shapes (chunks per lane,
// segments per half row, rows in flight) of the four projections; D, G:
// head dimension and query heads per KV head; NS: the split records the O
// phase merges per head.
template <int D, int G, int NS, int QCH, int QSEG, int QBUF, int OCH, int OSEG, int OBUF, int GCH, int GSEG, int GBUF,
          int DCH, int DSEG, int DBUF>
__global__ __launch_bounds__(kFThreads) void fused_layer_kernel(FusedArgs f) {
  using gemv::Mode;
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int blk = blockIdx.x, G_ = gridDim.x;
  const unsigned epoch = ld_cu(f.epoch) + 1u;
  float* stage = lds;  // phases 3-5: the projection's input
  const size_t stage_floats = ((size_t)f.stage_floats + 3) & ~size_t(3);
  float* gl = lds + stage_floats;  // phases 3-5: the GEMV body's LDS

  // ---- 1. RMSNorm1 + QKV -----------------------------------------------------
  {
    gemv::GemvBody<1, QCH, QSEG, QBUF, Mode::kNormQkv, QkvIO> body(f.qkv, QkvIO{}, lds, blk, G_, 0, tid);
    body.load_inputs();
    __builtin_amdgcn_sched_barrier(0);
    body.prime();
    body.run();
  }
  signal0(f, 0, epoch);

  // ---- 2. attention: item (KV head, split) of this block, four sub-bodies ---
  {
    using Body = attn::AttnBody<D, G, 1, false, kKvBf16, SubAttnIO<G>>;
    using Smem = typename Body::Smem;
    constexpr int RS = D + kPartLead;
    auto* sm = reinterpret_cast<Smem*>(lds);
    float* recs = lds + (kSub * sizeof(Smem) + 15) / 16 * 4;  // [kSub][G][RS]
    const int sb = tid / attn::kThreads, stid = tid % attn::kThreads;
    const int nsplit = f.attn.nsplit;
    const bool live = blk < f.attn_items;
    const int g = live ? blk / nsplit : 0, s = live ? blk % nsplit : 0;
    // sub-split s kSub + sb of kSub nsplit takes the split's tiles s kSub +
    // sb, + kSub nsplit, ...: the four together are split s's tiles
    Body body(f.attn, SubAttnIO<G>{recs + (size_t)sb * G * RS}, sm[sb], stid, s * kSub + sb, g, 0, live, nullptr, nullptr,
              nsplit * kSub);
    // K/V tiles do not depend on the QKV phase; the polling wave loads its
    // tiles after the wait, so its polls do not queue behind them
    if (wave != 0) body.prime();
    wait_phase(f, 0, epoch);
    if (wave == 0) body.prime();
    body.load_prologue();
    body.run(1.f, 1.f);
    __syncthreads();
    // wave 0: the four sub-splits' records -> split s's record (coherent)
    if (live && wave == 0) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float M = -INFINITY;
#pragma unroll
        for (int q = 0; q < kSub; ++q) M = fmaxf(M, recs[(q * G + h) * RS]);
        float fq[kSub], L = 0.f;
#pragma unroll
        for (int q = 0; q < kSub; ++q) {
          fq[q] = merge_factor(recs[(q * G + h) * RS], M);
          L = fmaf(recs[(q * G + h) * RS + 1], fq[q], L);
        }
        float* pr = f.attn.part + ((size_t)(g * G + h) * f.attn.nsplit_cap + s) * RS;
        for (int e = tid; e < D; e += kWave) {
          float O = 0.f;
#pragma unroll
          for (int q = 0; q < kSub; ++q) O = fmaf(recs[(q * G + h) * RS + kPartLead + e], fq[q], O);
          st_c(pr + kPartLead + e, O);
        }
        if (tid == 0) {
          st_c(pr, M);
          st_c(pr + 1, L);
        }
      }
    }
  }
  signal0(f, 1, epoch);

  // ---- 3. split merge + O projection + residual -------------------------------
  {
    gemv::GemvBody<1, OCH, OSEG, OBUF, Mode::kResidual, StageIO> body(f.oproj, StageIO{stage}, gl, blk, G_, 0, tid);
    if (wave != 0) body.prime();  // the polling wave prefetches after its wait
    body.load_resid();            // x, written before the launch
    wait_phase(f, 1, epoch);
    if (wave == 0) body.prime();
    // thread t: o elements 4t..4t+3 of one head, merged over its NS splits
    const int ns = f.attn.nsplit, nel = f.attn.n_heads * D;
    constexpr int RS = D + kPartLead;
    const int e = 4 * min(tid, nel / 4 - 1);
    const __amdgpu_buffer_rsrc_t pr =
        __builtin_amdgcn_make_buffer_rsrc((void*)f.attn.part, (short)0,
                                          f.attn.n_heads * f.attn.nsplit_cap * RS * (int)sizeof(float), 0x00020000);
    const unsigned ph = (unsigned)((e / D) * f.attn.nsplit_cap * RS);  // the head's first record, in floats
    float4 ov[NS];
    float ms[NS], ls[NS];
#pragma unroll
    for (int q = 0; q < NS; ++q) {
      const unsigned r = ph + (unsigned)(min(q, ns - 1) * RS);
      const float4 ml = ld_c4(pr, 4u * r);
      ms[q] = ml.x;
      ls[q] = ml.y;
      ov[q] = ld_c4(pr, 4u * (r + kPartLead + e % D));
    }
    float M = -INFINITY;
#pragma unroll
    for (int q = 0; q < NS; ++q)
      if (q < ns) M = fmaxf(M, ms[q]);
    float L = 0.f;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int q = 0; q < NS; ++q) {
      const float fq = q < ns ? merge_factor(ms[q], M) : 0.f;
      L = fmaf(ls[q], fq, L);
      acc.x = fmaf(ov[q].x, fq, acc.x);
      acc.y = fmaf(ov[q].y, fq, acc.y);
      acc.z = fmaf(ov[q].z, fq, acc.z);
      acc.w = fmaf(ov[q].w, fq, acc.w);
    }
    if (tid < nel / 4) {
      const float4 v = make_float4(acc.x / L, acc.y / L, acc.z / L, acc.w / L);
      *reinterpret_cast<float4*>(stage + e) = v;
      if (blk == 0) *reinterpret_cast<float4*>(f.attn.o + e) = v;  // the step's o (read after the launch)
    }
    __syncthreads();
    body.load_act();
    body.run();
  }
  signal0(f, 2, epoch);

  // ---- 4. RMSNorm2 + gate/up + siLu_Mul --------------------------------------
  {
    gemv::GemvBody<1, GCH, GSEG, GBUF, Mode::kGateUp, StageIO> body(f.gateup, StageIO{stage}, gl, blk, G_, 0, tid);
    if (wave != 0) body.prime();
    wait_phase(f, 2, epoch);
    if (wave == 0) body.prime();
    stage_in(stage, f.gateup.in_f32, f.gateup.din);
    body.load_inputs();
    body.run();
  }
  signal0(f, 3, epoch);

  // ---- 5. down projection + residual -> y --------------------------------------
  {
    gemv::GemvBody<1, DCH, DSEG, DBUF, Mode::kDownResidual, StageIO> body(f.down, StageIO{stage}, gl, blk, G_, 0,
                                                                         tid);
    if (wave != 0) body.prime();
    wait_phase(f, 3, epoch);
    if (wave == 0) body.prime();
    stage_in(stage, f.down.in_f32, f.down.din);
    body.load_inputs();
    body.run();
  }
  // the next launch's epoch: every block read this one at its start (each
  // waited for all blocks' phase-4 flags, so all have started)
  if (blk == 0) {
    wait_vm();
    __syncthreads();
    if (tid == 0) st_cu(f.epoch, epoch);
  }
}

template <int D, int G, int NS, int QCH, int QSEG, int QBUF, int OCH, int OSEG, int OBUF, int GCH, int GSEG, int GBUF,
          int DCH, int DSEG, int DBUF>
hipError_t launch_config(const FusedArgs& f, hipStream_t s, KernelEvents ev) {
  using Smem = attn::AttnSmem<D, G, kKvBf16>;
  using gemv::GemvBody;
  using gemv::Mode;
  const int G_ = kFusedGrid;
  const size_t stage = ((size_t)f.stage_floats + 3) & ~size_t(3);
  const size_t gl = std::max({GemvBody<1, OCH, OSEG, OBUF, Mode::kResidual, StageIO>::lds_floats(f.oproj.rows, G_),
                              GemvBody<1, GCH, GSEG, GBUF, Mode::kGateUp, StageIO>::lds_floats(f.gateup.rows, G_),
                              GemvBody<1, DCH, DSEG, DBUF, Mode::kDownResidual, StageIO>::lds_floats(f.down.rows,
                                                                                                     G_)});
  const size_t ql = GemvBody<1, QCH, QSEG, QBUF, Mode::kNormQkv, QkvIO>::lds_floats(f.qkv.rows, G_);
  const size_t attn = (kSub * sizeof(Smem) + 15) / 16 * 16 + (size_t)kSub * G * (D + kPartLead) * sizeof(float);
  const size_t lds = std::max({attn, (stage + gl) * sizeof(float), ql * sizeof(float)});
  if (lds > kMaxFusedLds || f.attn.nsplit > NS || f.attn_items > G_ || (f.attn.n_heads * D) % 4 != 0 ||
      f.attn.n_heads * D > 4 * kFThreads)
    return hipErrorInvalidValue;
  return ext_launch(
      fused_layer_kernel<D, G, NS, QCH, QSEG, QBUF, OCH, OSEG, OBUF, GCH, GSEG, GBUF, DCH, DSEG, DBUF>, dim3(G_),
      dim3(kFThreads), lds, s, ev, f);
}

}  // namespace

bool fused_layer_supported(const FusedShape& sh) {
  // the instantiated shape: the Phi-3-mini layer (d 96, MHA; projections of
  // 3072 inputs with 3 chunks per lane in 2 segments, the down projection's
  // 8192 inputs with 2 chunks in 8 segments)
  return sh.head_dim == 96 && sh.group == 1 && sh.q.maxch == 3 && sh.q.nseg_h == 2 && sh.o.maxch == 3 &&
         sh.o.nseg_h == 2 && sh.gu.maxch == 3 && sh.gu.nseg_h == 2 && sh.down.maxch == 2 && sh.down.nseg_h == 8;
}

int fused_layer_max_splits() { return kFusedMaxSplits; }
int fused_layer_grid() { return kFusedGrid; }

hipError_t launch_fused_layer(const FusedArgs& f, const FusedShape& sh, hipStream_t s, KernelEvents ev) {
  if (!fused_layer_supported(sh)) return hipErrorInvalidValue;
  // rows in flight per wave: the separate kernels' ring for QKV (the launch
  // starts with it), deeper rings where a phase's first rows are prefetched
  // ahead of a wait
  return launch_config<96, 1, kFusedMaxSplits, 3, 2, 1, 3, 2, 2, 3, 2, 2, 2, 8, 3>(f, s, ev);
}

}  // namespace fasttps
