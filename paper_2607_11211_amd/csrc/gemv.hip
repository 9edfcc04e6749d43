// Weight-streaming GEMV kernels of the decode layer (gfx950): the QKV
// projection with RMSNorm1, the O projection with the residual, the fused
// gate/up projection with RMSNorm2 and siLu_Mul, and the down projection with
// the residual and the bf16 rounding of y.
//
// At batch 1-8 the projections are matrix-vector products whose cost is the
// bf16 weight stream from HBM (Section 4.4 of the paper, OI and Accuracy: token-phase MLP and
// projections are bound by weight movement). Layout of the work:
//   * rows are dealt to the blocks round-robin (block b takes rows b, b + G,
//     b + 2G, ... of a grid of G blocks), so at any moment the chip reads a
//     compact window of the matrix;
//   * a row is cut into NSEG segments of 64 MAXCH 16-byte chunks; the W
//     waves of a block form W / NSEG groups of NSEG waves, wave (g, s) taking
//     segment s of the group's rows g, g + W / NSEG, ... Lane l of a wave
//     reads chunks l, l + 64, ... of its segment, so every load instruction
//     covers one contiguous kilobyte. W = 16 (one block per CU), or at one
//     sequence and rows of up to four segments W = 8 with two blocks per CU;
//   * each wave holds the activation values of its own chunks in registers
//     (fp32). At one sequence the block first stages the activation and the
//     gains in LDS (one load per 16 bytes per block, issued ahead of the
//     weight rows, the norm's sum of squares summed on the way) and the waves
//     read their chunks from there; otherwise each wave loads its chunks
//     itself before its first weight load. Only a row cut into segments
//     needs the block's waves to meet again, for its segment sums;
//   * each wave keeps NBUF rows in flight (2-4 KB): more outstanding loads
//     per CU only queue up in the memory system. With one row in flight the
//     next row's chunk j is issued right after chunk j is used, and the last
//     row issues nothing;
//   * every global load of the stream is issued unconditionally (clamped or
//     dead addresses where there is nothing to load), so the number of loads
//     in flight is the same on every path and the compiler waits for exactly
//     the ring slot a dot product needs.
// The gate/up projection reads the interlaced W_gu (Section 3.2 item 1,
// Alg. 4) with tiles of one row: row 2k is gate row k and row 2k+1 up row k,
// so one row of this kernel is the pair [gate k | up k] of 2D values, its two
// halves are the kernel's two segment halves, and siLu_Mul (Eq. 30-31)
// combines them in LDS.
#include "gemv_body.h"

namespace fasttps {

namespace {

using gemv::halves;
using gemv::has_residual;
using gemv::kNumCu;
using gemv::kWaves;
using gemv::max_chunks;
using gemv::Mode;
using gemv::segments_for;

// floats before the input stage in a staged kernel's LDS (16-byte aligned)
__host__ __device__ constexpr size_t staged_offset(size_t body_floats) { return (body_floats + 3) / 4 * 4; }
// the largest LDS a staged launch takes (beyond it the waves load their own inputs)
constexpr size_t kMaxStagedLds = 64 * 1024;
// waves per block of the staged kernel where the row's segments fit (else 16)
constexpr int kStagedWaves = 8;

template <int BT, int MAXCH, int NSEG_H, int NBUF, Mode MODE>
__global__ __launch_bounds__(kWaves * kWave) void gemv_kernel(GemvArgs a) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  gemv::GemvBody<BT, MAXCH, NSEG_H, NBUF, MODE, gemv::GlobalIO> body(a, gemv::GlobalIO{}, lds, blockIdx.x, gridDim.x,
                                                                    blockIdx.y * BT, threadIdx.x);
  body.load_inputs();
  __builtin_amdgcn_sched_barrier(0);  // keep these loads ahead of the weight loads
  body.prime();
  body.run();
}

// One sequence with its inputs staged in LDS: the block loads the activation
// and the gains once (InputStage), issues its first weight rows behind them,
// and its waves take their chunks from the stage; the norm's sum of squares
// is summed while the stage is stored (one block barrier for both). Blocks of
// WAVES waves; with 8, two blocks share a CU (at most 128 registers a lane).
template <int MAXCH, int NSEG_H, int NBUF, Mode MODE, int WAVES>
__global__ __launch_bounds__(WAVES* kWave) __attribute__((amdgpu_waves_per_eu(4, 8))) void gemv_staged_kernel(
    GemvArgs a) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  using Body = gemv::GemvBody<1, MAXCH, NSEG_H, NBUF, MODE, gemv::GlobalIO, WAVES>;
  Body body(a, gemv::GlobalIO{}, lds, blockIdx.x, gridDim.x, 0, threadIdx.x);
  float* wss = lds + staged_offset(Body::lds_floats(a.rows, gridDim.x));  // [WAVES]
  v4u* stage = reinterpret_cast<v4u*>(wss + 16);
  gemv::InputStage<MODE, WAVES> st;
  st.load(a, threadIdx.x);
  body.load_resid();
  __builtin_amdgcn_sched_barrier(0);  // keep these loads ahead of the weight loads
  body.prime();
  st.store(stage, wss);
  __syncthreads();
  body.load_act_lds(stage, wss);
  body.run();
}

// Launch shape: a batch tile of BT sequences, MAXCH chunks per lane and row
// segment, NSEG_H segments per half row, gemv::ring_rows rows in flight per
// wave (2-4 KB: at this size the memory system's queues stay short enough
// that the waves that start last do not finish much later than the rest).
template <int BT, int MAXCH, int NSEG_H, Mode MODE>
hipError_t launch_shape(const GemvArgs& a, hipStream_t s, KernelEvents ev) {
  constexpr int NBUF = gemv::ring_rows(BT, MAXCH);
  const int nblk = a.rows < kNumCu ? a.rows : kNumCu;
  // unsegmented rows add the residual from the register copy only
  constexpr int NG = kWaves / (halves<MODE>() * NSEG_H);
  if (halves<MODE>() * NSEG_H == 1 && has_residual<MODE>() &&
      BT * ((((a.rows + nblk - 1) / nblk) + NG - 1) / NG) > kWave)
    return hipErrorInvalidValue;
  dim3 grid(nblk, (a.batch + BT - 1) / BT);
  const size_t body_floats = (size_t)halves<MODE>() * NSEG_H * BT * ((a.rows + nblk - 1) / nblk) + (size_t)NSEG_H * BT;
  if constexpr (BT == 1 && MODE != Mode::kPlain) {
    constexpr int W2 = kStagedWaves;
    if constexpr (halves<MODE>() * NSEG_H <= W2 / 2) {
      using Stage = gemv::InputStage<MODE, W2>;
      const int nblk2 = a.rows < kNumCu * (kWaves / W2) ? a.rows : kNumCu * (kWaves / W2);
      const size_t bf2 =
          (size_t)halves<MODE>() * NSEG_H * ((a.rows + nblk2 - 1) / nblk2) + (size_t)NSEG_H;
      const size_t lds = (staged_offset(bf2) + 16) * sizeof(float) + (size_t)Stage::pieces(a.din) * sizeof(v4u);
      constexpr int NG2 = W2 / (halves<MODE>() * NSEG_H);
      const bool resid_ok = !(halves<MODE>() * NSEG_H == 1 && has_residual<MODE>() &&
                              (((a.rows + nblk2 - 1) / nblk2) + NG2 - 1) / NG2 > kWave);
      if (Stage::fits(a.din) && lds <= kMaxStagedLds && resid_ok)
        return ext_launch(gemv_staged_kernel<MAXCH, NSEG_H, NBUF, MODE, W2>, dim3(nblk2), dim3(W2 * kWave), lds, s,
                          ev, a);
    }
    using Stage = gemv::InputStage<MODE, kWaves>;
    const size_t lds = (staged_offset(body_floats) + 16) * sizeof(float) + (size_t)Stage::pieces(a.din) * sizeof(v4u);
    if (Stage::fits(a.din) && lds <= kMaxStagedLds)
      return ext_launch(gemv_staged_kernel<MAXCH, NSEG_H, NBUF, MODE, kWaves>, grid, dim3(kWaves * kWave), lds, s,
                        ev, a);
  }
  const size_t lds = body_floats * sizeof(float);
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

// ---- the O projection with the split merge in its prologue (batch 1) ------

// the activation from an LDS stage
struct StageIO {
  const float* stage;
  __device__ __forceinline__ float4 act4(const GemvArgs& a, int b, int i4) const {
    return reinterpret_cast<const float4*>(stage + (size_t)b * a.din)[i4];
  }
  __device__ __forceinline__ float res(const GemvArgs& a, size_t o) const { return a.res_f32[o]; }
  __device__ __forceinline__ void out(const GemvArgs& a, size_t o, float v) const { a.out[o] = v; }
};

constexpr int kMergeThreads = kWaves * kWave;
// rows in flight per wave: one, as in the separate O projection (two or
// three, the block's whole share of W_o primed before the merge, were slower
// on MI355X: the Phi-3 layer step 59.0 -> 59.6 and 60.4 us)
constexpr int kMergeRing = 1;
static_assert(kMergeMaxElems <= 4 * kMergeThreads, "four o elements per thread");

// Every block: (1) loads, for its thread's four elements of o, the partial o
// values and the (m, l) of every split of their head, then issues its first
// weight rows; (2) merges the splits (M = max m, factors e^(m - M),
// L = sum l e^(m - M), o = sum o e^(m - M) / L, as the combine kernel does)
// into the LDS stage, with no block barrier until the stage is complete; (3)
// streams its W_o rows against the stage with the residual added.
template <int MAXCH, int NSEG_H, int NS>
__global__ __launch_bounds__(kMergeThreads) void oproj_merge_kernel(GemvArgs a, MergeArgs m) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  constexpr int NBUF = kMergeRing;
  const int tid = threadIdx.x;
  const int D = m.head_dim, ns = m.nsplit, nel = m.n_heads * D;
  const int rs = D + kPartLead;  // floats per split record
  float* stage = lds;            // o [H d]
  float* gl = lds + nel;

  // (1) the partials (o is 16-byte aligned in every record and D is a
  // multiple of 4, so the four elements share a head); threads past the last
  // element load nothing (whole waves of them skip the loads)
  const bool has_e = tid < nel / 4;
  const int e = 4 * min(tid, nel / 4 - 1);
  const float* ph = m.part + (size_t)(e / D) * m.nsplit_cap * rs;
  float4 ov[NS];
  float2 ml[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    ml[s] = make_float2(0.f, 0.f);
    ov[s] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  if (has_e) {
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const float* r = ph + (size_t)min(s, ns - 1) * rs;
      ml[s] = *reinterpret_cast<const float2*>(r);
      ov[s] = *reinterpret_cast<const float4*>(r + kPartLead + e % D);
    }
  }
  gemv::GemvBody<1, MAXCH, NSEG_H, NBUF, Mode::kResidual, StageIO> body(a, StageIO{stage}, gl, blockIdx.x, gridDim.x,
                                                                        0, tid);
  body.load_resid();
  __builtin_amdgcn_sched_barrier(0);  // the weight loads go out after the partials' and the residual's
  body.prime();

  // (2) the merge of this thread's head
  float M = -INFINITY;
#pragma unroll
  for (int s = 0; s < NS; ++s)
    if (s < ns) M = fmaxf(M, ml[s].x);
  float L = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const float f = s < ns ? merge_factor(ml[s].x, M) : 0.f;
    L = fmaf(ml[s].y, f, L);
    acc.x = fmaf(ov[s].x, f, acc.x);
    acc.y = fmaf(ov[s].y, f, acc.y);
    acc.z = fmaf(ov[s].z, f, acc.z);
    acc.w = fmaf(ov[s].w, f, acc.w);
  }
  if (has_e) {
    const float4 v = make_float4(acc.x / L, acc.y / L, acc.z / L, acc.w / L);
    *reinterpret_cast<float4*>(stage + e) = v;
    if (blockIdx.x == 0) *reinterpret_cast<float4*>(m.o + e) = v;
  }
  __syncthreads();

  // (3) the projection
  body.load_act();
  body.run();
}

template <int MAXCH, int NSEG_H>
hipError_t launch_merge_shape(const GemvArgs& a, const MergeArgs& m, hipStream_t s, KernelEvents ev) {
  using Body = gemv::GemvBody<1, MAXCH, NSEG_H, kMergeRing, Mode::kResidual, StageIO>;
  const int nblk = a.rows < kNumCu ? a.rows : kNumCu;
  constexpr int NG = kWaves / NSEG_H;
  if (NSEG_H == 1 && (((a.rows + nblk - 1) / nblk) + NG - 1) / NG > kWave) return hipErrorInvalidValue;
  const size_t lds = ((size_t)m.n_heads * m.head_dim + Body::lds_floats(a.rows, nblk)) * sizeof(float);
  if (m.nsplit <= 4)
    return ext_launch(oproj_merge_kernel<MAXCH, NSEG_H, 4>, dim3(nblk), dim3(kMergeThreads), lds, s, ev, a, m);
  if (m.nsplit <= 8)
    return ext_launch(oproj_merge_kernel<MAXCH, NSEG_H, 8>, dim3(nblk), dim3(kMergeThreads), lds, s, ev, a, m);
  return ext_launch(oproj_merge_kernel<MAXCH, NSEG_H, 16>, dim3(nblk), dim3(kMergeThreads), lds, s, ev, a, m);
}

template <int MAXCH>
hipError_t launch_merge_seg(const GemvArgs& a, const MergeArgs& m, int nseg_h, hipStream_t s, KernelEvents ev) {
  switch (nseg_h) {
    case 1: return launch_merge_shape<MAXCH, 1>(a, m, s, ev);
    case 2: return launch_merge_shape<MAXCH, 2>(a, m, s, ev);
    case 4: return launch_merge_shape<MAXCH, 4>(a, m, s, ev);
    default: return hipErrorInvalidValue;
  }
}

// the shape launch_bt<1, kResidual> picks for din inputs (chunks per lane,
// segments per half row), restricted to what the merge kernel instantiates
bool merge_shape(int din, int* maxch, int* nseg_h) {
  const int nch = din / 8;
  const int ns = segments_for(din, max_chunks(1, false));
  if (ns > kWaves) return false;
  const int per = (nch + ns * kWave - 1) / (ns * kWave);
  if (per > 3 || ns > 4) return false;
  *maxch = per < 1 ? 1 : per;
  *nseg_h = ns;
  return true;
}

}  // namespace

bool oproj_merge_supported(int n_heads, int head_dim, int nsplit, int rows) {
  int mc, sg;
  const int nel = n_heads * head_dim;
  return nsplit >= 1 && nsplit <= kMergeMaxSplits && nel <= kMergeMaxElems && head_dim % 4 == 0 &&
         merge_shape(nel, &mc, &sg) && rows >= 1;
}

hipError_t launch_oproj_merge(const GemvArgs& a, const MergeArgs& m, hipStream_t s, KernelEvents ev) {
  if (a.batch != 1 || !oproj_merge_supported(m.n_heads, m.head_dim, m.nsplit, a.rows) ||
      a.din != m.n_heads * m.head_dim)
    return hipErrorInvalidValue;
  int maxch, nseg_h;
  merge_shape(a.din, &maxch, &nseg_h);
  switch (maxch) {
    case 1: return launch_merge_seg<1>(a, m, nseg_h, s, ev);
    case 2: return launch_merge_seg<2>(a, m, nseg_h, s, ev);
    case 3: return launch_merge_seg<3>(a, m, nseg_h, s, ev);
    default: return hipErrorInvalidValue;
  }
}

FusedShape::Gemv gemv_shape_b1(int din, bool gate_up) {
  const int nh = gate_up ? 2 : 1;
  const int nch = din / 8;
  int cap = max_chunks(1, false);
  if (segments_for(din, cap) * nh > kWaves) cap = max_chunks(1, true);
  const int nseg_h = segments_for(din, cap);
  const int per = (nch + nseg_h * kWave - 1) / (nseg_h * kWave);
  const int maxch = per <= 1 ? 1 : per <= 2 ? 2 : per <= 3 ? 3 : per <= 4 ? 4 : 6;
  return {maxch, nseg_h, gemv::ring_rows(1, maxch)};
}

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
