// The whole decode step of one sequence as one persistent kernel (gfx950).
//
// Six kernels per layer step cost about 3 us each at their boundaries (launch,
// first loads, the last waves), a third of the Phi-3 layer's time, while the
// weight streams themselves already run at the chip's read rate. Here one
// grid of 256 blocks x 16 waves (one block per CU) runs the six phases of the
// step in turn: RMSNorm1 + QKV, attention splits (RoPE, append, partial
// softmax), the split merge, O projection + residual, RMSNorm2 + gate/up +
// siLu_Mul, down projection + residual. The paper's pipeline overlaps weight
// loads with computation inside an operator (Section 3.2 item 3); here the
// overlap also crosses the operators: a block that finishes a phase issues the
// first weight rows (or K/V tiles) of the next phase before it waits for the
// phase's input, so the wait and the memory system's ramp overlap.
//
// Phase hand-over between blocks (L2 caches are per XCD and not coherent):
//   * data a later phase reads in another block (q|k|v, the split partials,
//     o, h1, the MLP activation) is written with agent-coherent stores and
//     read with agent-coherent loads (global_store / global_load sc1, the
//     accesses of relaxed agent-scope atomics), so no L2 write-back or
//     invalidate is needed;
//   * a block ends a phase with all its stores complete (s_waitcnt vmcnt(0)
//     in every wave, then a block barrier) and one coherent store of the
//     launch's epoch into its flag of that phase;
//   * wave 0 of every block polls the 256 flags of the phase it needs
//     (coherent loads) until all hold the epoch, then the block's barrier
//     releases the other waves, whose weight loads are already in flight.
// Measured on MI355X (Phi-3 layer, KV 4096): 85 us per step against 62 us for
// the six separate kernels replayed from a HIP graph. Per-block wall-clock
// stamps show the phases themselves as fast as the separate kernels (gate/up
// faster), but each hand-over costs 2-9 us: the flag round trips through
// coherent memory are slow under load, and a block's polling loads queue
// behind the weight or K/V loads its waves issued ahead of the wait (a CU
// serves its vector memory loads in order). The path is kept as an
// alternative (FASTTPS_GEMM_FUSED), not the default.
// Every wait is bounded: past kSpinLimit polls the block counts an error
// (read through the debug hook) and goes on, so a grid that cannot be fully
// resident ends instead of hanging. The epoch lives in device memory and is
// advanced by block 0 at its end, so replays of a captured graph get fresh
// epochs.
#include "attn_body.h"
#include "gemv_body.h"

#include <algorithm>

namespace fasttps {

namespace {

constexpr int kFThreads = 1024;
constexpr int kSubBlocks = kFThreads / attn::kThreads;  // attention items per block and round
constexpr long kSpinLimit = 1L << 18;
constexpr size_t kMaxFusedLds = 160 * 1024;
constexpr int kFusedGrid = 256;                      // one block per CU
constexpr int kFlagsPerLane = kFusedGrid / kWave;     // a wave polls the grid's flags

// GEMV IO of the fused kernel: activation from the LDS stage, residual and
// fp32 outputs coherent
struct FusedGemvIO {
  const float* stage;  // LDS
  __device__ __forceinline__ float4 act4(const GemvArgs& a, int b, int i4) const {
    return reinterpret_cast<const float4*>(stage + (size_t)b * a.din)[i4];
  }
  __device__ __forceinline__ float res(const GemvArgs&, size_t o) const { return 0.f; }
  __device__ __forceinline__ void out(const GemvArgs& a, size_t o, float v) const { st_c(a.out + o, v); }
};
struct FusedGemvResIO : FusedGemvIO {
  __device__ __forceinline__ float res(const GemvArgs& a, size_t o) const { return ld_c(a.res_f32 + o); }
};
struct FusedAttnIO {
  __device__ __forceinline__ float qkv(const AttnArgs& a, size_t i) const { return ld_c(a.qkv + i); }
  __device__ __forceinline__ void part(float* p, float v) const { st_c(p, v); }
};

// this block's stores of phase `ph` are complete: publish its flag
__device__ __forceinline__ void signal(const FusedArgs& f, int ph, unsigned epoch) {
  wait_vm();
  __syncthreads();
  if (threadIdx.x == 0) st_cu(f.flags + (size_t)ph * gridDim.x + blockIdx.x, epoch);
}

// every block's flag of phase `ph` holds the epoch (wave 0 polls; the block
// barrier then releases the other waves)
__device__ __forceinline__ void wait_phase(const FusedArgs& f, int ph, unsigned epoch, int wave) {
  if (wave == 0) {
    const unsigned* fl = f.flags + (size_t)ph * gridDim.x;
    const int lane = threadIdx.x & (kWave - 1);
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
// head dimension and query heads per KV head.
template <int D, int G, int QCH, int QSEG, int QBUF, int OCH, int OSEG, int OBUF, int GCH, int GSEG, int GBUF,
          int DCH, int DSEG, int DBUF>
__global__ __launch_bounds__(kFThreads) void fused_layer_kernel(FusedArgs f) {
  using gemv::Mode;
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int blk = blockIdx.x, G_ = gridDim.x;
  const unsigned epoch = ld_cu(f.epoch) + 1u;
  float* stage = lds;  // phases 4-6: the activation; then the GEMV's LDS
  const size_t stage_floats = ((size_t)f.stage_floats + 3) & ~size_t(3);

  // ---- 1. RMSNorm1 + QKV -----------------------------------------------------
  {
    gemv::GemvBody<1, QCH, QSEG, QBUF, Mode::kNormQkv, FusedGemvIO> body(f.qkv, FusedGemvIO{stage}, lds, blk, G_, 0,
                                                                        tid);
    body.load_inputs();
    __builtin_amdgcn_sched_barrier(0);
    body.prime();
    body.run();
  }
  signal(f, 0, epoch);

  // ---- 2. attention splits: four 256-thread items per block and round ------
  {
    using Body = attn::AttnBody<D, G, 1, false, kKvBf16, FusedAttnIO>;
    auto* sm = reinterpret_cast<typename Body::Smem*>(lds);
    const int sb = tid / attn::kThreads, stid = tid % attn::kThreads;
    const int nkv = f.attn.n_kv_heads;
    const int rounds = (f.attn_items + G_ * kSubBlocks - 1) / (G_ * kSubBlocks);
    for (int rd = 0; rd < rounds; ++rd) {
      const int it = (rd * kSubBlocks + sb) * G_ + blk;  // items dealt over the blocks first
      const bool live = it < f.attn_items;
      const int itc = live ? it : 0;
      Body body(f.attn, FusedAttnIO{}, sm[sb], stid, itc / nkv, itc % nkv, 0, live);
      // K/V tiles do not depend on the QKV phase; the polling wave loads its
      // tiles after the wait, so its polls do not queue behind them
      if (rd > 0 || wave != 0) body.prime();
      if (rd == 0) {
        wait_phase(f, 0, epoch, wave);
        if (wave == 0) body.prime();
      }
      body.load_prologue();
      body.run(1.f, 1.f);
    }
  }
  signal(f, 1, epoch);

  // ---- 3. merge the splits: every block merges a contiguous slice of o ----
  // (o element i of head i / D needs split s's o value and its (m, l), for
  // every split: one round trip of loads, then LDS sums)
  {
    const int nsplit = f.attn.nsplit, D_ = D;
    const int nel = f.attn.n_heads * D_;
    const int per = (nel + G_ - 1) / G_;               // elements of this block
    const int e0 = blk * per;
    const int t = tid;
    const bool act = t < per * nsplit;
    const int el = min(e0 + (act ? t / nsplit : 0), nel - 1), sp = act ? t % nsplit : 0;
    const int h = el / D_, e = el % D_;
    const float* pr = f.attn.part + ((size_t)h * f.attn.nsplit_cap + sp) * (D + kPartLead);
    float* mm = stage;                                 // [per][64] m, then l, then o of each split
    float* ll = stage + (size_t)per * kWave;
    float* oo = stage + 2 * (size_t)per * kWave;
    wait_phase(f, 1, epoch, wave);
    const float mv = ld_c(pr), lv = ld_c(pr + 1), ov = ld_c(pr + kPartLead + e);
    if (act) {
      const int r = t / nsplit;
      mm[r * kWave + sp] = mv;
      ll[r * kWave + sp] = lv;
      oo[r * kWave + sp] = ov;
    }
    __syncthreads();
    if (t < per && e0 + t < nel) {
      float M = -INFINITY;
      for (int q = 0; q < nsplit; ++q) M = fmaxf(M, mm[t * kWave + q]);
      float L = 0.f, O = 0.f;
      for (int q = 0; q < nsplit; ++q) {
        const float fq = attn::merge_factor(mm[t * kWave + q], M);
        L = fmaf(ll[t * kWave + q], fq, L);
        O = fmaf(oo[t * kWave + q], fq, O);
      }
      st_c(f.attn.o + e0 + t, O / L);
    }
  }
  signal(f, 2, epoch);

  // ---- 4. O projection + residual --------------------------------------------
  {
    gemv::GemvBody<1, OCH, OSEG, OBUF, Mode::kResidual, FusedGemvIO> body(f.oproj, FusedGemvIO{stage},
                                                                         lds + stage_floats, blk, G_, 0, tid);
    if (wave != 0) body.prime();  // the polling wave prefetches after its wait
    wait_phase(f, 2, epoch, wave);
    if (wave == 0) body.prime();
    stage_in(stage, f.oproj.in_f32, f.oproj.din);
    body.load_inputs();
    body.run();
  }
  signal(f, 3, epoch);

  // ---- 5. RMSNorm2 + gate/up + siLu_Mul --------------------------------------
  {
    gemv::GemvBody<1, GCH, GSEG, GBUF, Mode::kGateUp, FusedGemvIO> body(f.gateup, FusedGemvIO{stage},
                                                                       lds + stage_floats, blk, G_, 0, tid);
    if (wave != 0) body.prime();  // the polling wave prefetches after its wait
    wait_phase(f, 3, epoch, wave);
    if (wave == 0) body.prime();
    stage_in(stage, f.gateup.in_f32, f.gateup.din);
    body.load_inputs();
    body.run();
  }
  signal(f, 4, epoch);

  // ---- 6. down projection + residual -> y --------------------------------------
  {
    gemv::GemvBody<1, DCH, DSEG, DBUF, Mode::kDownResidual, FusedGemvResIO> body(
        f.down, FusedGemvResIO{{stage}}, lds + stage_floats, blk, G_, 0, tid);
    if (wave != 0) body.prime();  // the polling wave prefetches after its wait
    wait_phase(f, 4, epoch, wave);
    if (wave == 0) body.prime();
    stage_in(stage, f.down.in_f32, f.down.din);
    body.load_inputs();
    body.run();
  }
  // the next launch's epoch: every block read this one at its start (each
  // waited for all blocks' phase-5 flags, so all have started)
  if (blk == 0) {
    wait_vm();
    __syncthreads();
    if (tid == 0) st_cu(f.epoch, epoch);
  }
}

template <int D, int G, int QCH, int QSEG, int QBUF, int OCH, int OSEG, int OBUF, int GCH, int GSEG, int GBUF,
          int DCH, int DSEG, int DBUF>
hipError_t launch_config(const FusedArgs& f, hipStream_t s, KernelEvents ev) {
  using Smem = attn::AttnSmem<D, G, kKvBf16>;
  using gemv::GemvBody;
  using gemv::Mode;
  const int G_ = kFusedGrid;
  const size_t stage = ((size_t)f.stage_floats + 3) & ~size_t(3);
  const size_t gl = std::max({GemvBody<1, OCH, OSEG, OBUF, Mode::kResidual, FusedGemvIO>::lds_floats(f.oproj.rows, G_),
                              GemvBody<1, GCH, GSEG, GBUF, Mode::kGateUp, FusedGemvIO>::lds_floats(f.gateup.rows, G_),
                              GemvBody<1, DCH, DSEG, DBUF, Mode::kDownResidual, FusedGemvIO>::lds_floats(f.down.rows,
                                                                                                      G_)});
  const size_t ql = GemvBody<1, QCH, QSEG, QBUF, Mode::kNormQkv, FusedGemvIO>::lds_floats(f.qkv.rows, G_);
  const int per = (f.attn.n_heads * D + G_ - 1) / G_;
  const size_t merge = 3 * (size_t)per * kWave;
  const size_t lds =
      std::max({(size_t)kSubBlocks * sizeof(Smem), (stage + gl) * sizeof(float), ql * sizeof(float),
                merge * sizeof(float)});
  if (lds > kMaxFusedLds || f.attn.nsplit > kWave || per * f.attn.nsplit > kFThreads)
    return hipErrorInvalidValue;
  return ext_launch(fused_layer_kernel<D, G, QCH, QSEG, QBUF, OCH, OSEG, OBUF, GCH, GSEG, GBUF, DCH, DSEG, DBUF>,
                    dim3(G_), dim3(kFThreads), lds, s, ev, f);
}

}  // namespace

bool fused_layer_supported(const FusedShape& sh) {
  // the instantiated shape: the Phi-3-mini layer (d 96, MHA; projections of
  // 3072 inputs with 3 chunks per lane in 2 segments, the down projection's
  // 8192 inputs with 2 chunks in 8 segments), each with the ring depth of the
  // separate GEMV kernel
  return sh.head_dim == 96 && sh.group == 1 && sh.q == FusedShape::Gemv{3, 2, 1} && sh.o == FusedShape::Gemv{3, 2, 1} &&
         sh.gu == FusedShape::Gemv{3, 2, 1} && sh.down == FusedShape::Gemv{2, 8, 1};
}

hipError_t launch_fused_layer(const FusedArgs& f, const FusedShape& sh, hipStream_t s, KernelEvents ev) {
  if (!fused_layer_supported(sh)) return hipErrorInvalidValue;
  return launch_config<96, 1, 3, 2, 1, 3, 2, 1, 3, 2, 1, 2, 8, 1>(f, s, ev);
}

}  // namespace fasttps
