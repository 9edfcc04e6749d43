// The fused MLP of the decode layer with the intermediate kept on chip
// (Section 3.2 "Fusion MLP", Alg. 4, Eq. 29-32): one kernel computes, per
// block, the gate/up projection of a slice of the intermediate units with
// RMSNorm2 and siLu_Mul, keeps that slice of h^sm in LDS, and multiplies it
// with the matching columns of W_down into a partial of y; a second kernel
// adds the partials of all blocks in a fixed order, with the residual, and
// rounds y to bf16.
//
// Block b of G takes the units k = b, b + G, b + 2G, ... (the rows the GEMV
// body deals it), so its gate/up rows stream exactly as in the separate
// gate/up kernel. W_down is packed for this kernel as G slices [D][U8]:
// slice b holds W_down[d, b + G i] at [d][i] (i < U8 = the units per block
// rounded up to a multiple of 8, zero past K), so a block's down-projection
// weights are one contiguous run of D U8 values and thread t's output rows
// d = t, t + 1024, ... each read U8 contiguous values.
//
// Alg. 4 stores h^sm to L3 and loads it again for the down projection; here
// it never leaves the CU. The price is the partial sums of y: G x B x D fp32
// written and read back by the second kernel.
#include "gemv_body.h"

namespace fasttps {

namespace {

using gemv::kNumCu;
using gemv::kWaves;
using gemv::max_chunks;
using gemv::Mode;
using gemv::segments_for;

constexpr int kThreads = kWaves * kWave;

// gate/up outputs go to the block's LDS slice of h^sm: a[s][i] for sequence
// s of the batch tile and block-local unit i
struct SliceIO {
  float* a_lds;
  int b0, blk, G, u8;
  __device__ __forceinline__ float4 act4(const GemvArgs& a, int b, int i4) const {
    return reinterpret_cast<const float4*>(a.in_f32 + (size_t)b * a.din)[i4];
  }
  __device__ __forceinline__ float res(const GemvArgs&, size_t) const { return 0.f; }
  __device__ __forceinline__ void out(const GemvArgs& a, size_t o, float v) const {
    const int s = (int)(o / a.rows) - b0;
    const int i = ((int)(o % a.rows) - blk) / G;
    a_lds[s * u8 + i] = v;
  }
};

template <int BT, int MAXCH, int NSEG_H, int NBUF>
__global__ __launch_bounds__(kThreads) void mlp_fused_kernel(GemvArgs a, MlpFusedArgs m) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  using Body = gemv::GemvBody<BT, MAXCH, NSEG_H, NBUF, Mode::kGateUp, SliceIO>;
  const int blk = blockIdx.x, G = gridDim.x, b0 = blockIdx.y * BT;
  const int tid = threadIdx.x;
  float* a_lds = lds + Body::lds_floats(a.rows, G);
  // units past the block's rows stay zero (their packed W_down columns are
  // zero too, and 0 * 0 keeps the sums clean)
  for (int t = tid; t < BT * m.u8; t += kThreads) a_lds[t] = 0.f;
  Body body(a, SliceIO{a_lds, b0, blk, G, m.u8}, lds, blk, G, b0, tid);
  body.load_inputs();
  __builtin_amdgcn_sched_barrier(0);  // keep these loads ahead of the weight loads
  body.prime();
  body.run();
  __syncthreads();  // the slice of h^sm is complete

  // down projection of the slice: y_part[s][d] = sum_i a[s][i] W_down[d, blk + G i],
  // one output row per thread at a time, its u8 values in order. (Loading
  // two rows' chunks in groups of eight, 16 loads in flight per thread, made
  // the Phi-3 kernel slower on MI355X: 31.7 against 27.2 us.)
  const int nb = min(BT, a.batch - b0);
  const int cpr = m.u8 / 8;  // 16-byte chunks per output row
  const v4u* Wd = reinterpret_cast<const v4u*>(m.w_down_slices) + (size_t)blk * m.hidden * cpr;
  for (int d = tid; d < m.hidden; d += kThreads) {
    float acc[BT];
#pragma unroll
    for (int s = 0; s < BT; ++s) acc[s] = 0.f;
    const v4u* row = Wd + (size_t)d * cpr;
    for (int c = 0; c < cpr; ++c) {
      float w[8];
      unpack8(row[c], w);
#pragma unroll
      for (int s = 0; s < BT; ++s) {
        const float* as = a_lds + s * m.u8 + 8 * c;
        float t = acc[s];
#pragma unroll
        for (int e = 0; e < 8; ++e) t = fmaf(w[e], as[e], t);
        acc[s] = t;
      }
    }
#pragma unroll
    for (int s = 0; s < BT; ++s)
      if (s < nb) m.part[((size_t)blk * m.batch + b0 + s) * m.hidden + d] = acc[s];
  }
}

// y[s][d] = bf16(h1[s][d] + sum_b part[b][s][d]), the blocks' partials added
// in a fixed order: thread (g, j) of a block of 256 adds the partials b = g,
// g + 16, ... of output j of the block's 16 (all its loads issued at once),
// then the 16 groups are added in order.
constexpr int kRedOut = 16;                    // outputs per block
constexpr int kGroups = 256 / kRedOut;         // threads per output
constexpr int kRedLoads = 16;                  // partials per thread (256 slices at most)
static_assert(kGroups * kRedLoads >= 256, "one round of loads covers every slice");
__global__ __launch_bounds__(256) void mlp_reduce_kernel(MlpFusedArgs m, const float* __restrict__ h1,
                                                         uint16_t* __restrict__ y) {
  __shared__ float red[kGroups][kRedOut];
  const int tid = threadIdx.x;
  const int j = tid % kRedOut, g = tid / kRedOut;
  const int s = blockIdx.y;
  const int d = min(blockIdx.x * kRedOut + j, m.hidden - 1);
  float v[kRedLoads];
#pragma unroll
  for (int i = 0; i < kRedLoads; ++i)
    v[i] = m.part[((size_t)min(g + kGroups * i, m.nblk - 1) * m.batch + s) * m.hidden + d];
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < kRedLoads; ++i)
    if (g + kGroups * i < m.nblk) t += v[i];
  red[g][j] = t;
  __syncthreads();
  if (g == 0 && blockIdx.x * kRedOut + j < m.hidden) {
    float u = 0.f;
#pragma unroll
    for (int q = 0; q < kGroups; ++q) u += red[q][j];
    y[(size_t)s * m.hidden + d] = f32_to_bf16(h1[(size_t)s * m.hidden + d] + u);
  }
}

// W_down [D, K] -> G slices [D][u8]: slice b, row d, column i = W_down[d, b + G i]
__global__ __launch_bounds__(256) void pack_down_slices_kernel(const uint16_t* __restrict__ wd,
                                                               uint16_t* __restrict__ dst, int hidden, int inter,
                                                               int G, int u8) {
  const int b = blockIdx.x, d = blockIdx.y;
  for (int i = threadIdx.x; i < u8; i += blockDim.x) {
    const int k = b + G * i;
    dst[((size_t)b * hidden + d) * u8 + i] = k < inter ? wd[(size_t)d * inter + k] : (uint16_t)0;
  }
}

template <int BT, int MAXCH, int NSEG_H>
hipError_t launch_shape(const GemvArgs& a, const MlpFusedArgs& m, hipStream_t s, KernelEvents ev) {
  constexpr int NBUF = gemv::ring_rows(BT, MAXCH);
  using Body = gemv::GemvBody<BT, MAXCH, NSEG_H, NBUF, Mode::kGateUp, SliceIO>;
  dim3 grid(m.nblk, (a.batch + BT - 1) / BT);
  const size_t lds = (Body::lds_floats(a.rows, m.nblk) + (size_t)BT * m.u8) * sizeof(float);
  if (lds > 64 * 1024) return hipErrorInvalidValue;
  return ext_launch(mlp_fused_kernel<BT, MAXCH, NSEG_H, NBUF>, grid, dim3(kThreads), lds, s, ev, a, m);
}

template <int BT, int MAXCH>
hipError_t launch_seg(const GemvArgs& a, const MlpFusedArgs& m, int nseg_h, hipStream_t s, KernelEvents ev) {
  switch (nseg_h) {
    case 1: return launch_shape<BT, MAXCH, 1>(a, m, s, ev);
    case 2: return launch_shape<BT, MAXCH, 2>(a, m, s, ev);
    case 4: return launch_shape<BT, MAXCH, 4>(a, m, s, ev);
    case 8: return launch_shape<BT, MAXCH, 8>(a, m, s, ev);
    default: return hipErrorInvalidValue;
  }
}

// the gate/up projection's launch shape, as in the separate gate/up kernel
template <int BT>
hipError_t launch_bt(const GemvArgs& a, const MlpFusedArgs& m, hipStream_t s, KernelEvents ev) {
  const int nch = a.din / 8;
  int cap = max_chunks(BT, false);
  if (segments_for(a.din, cap) * 2 > kWaves) cap = max_chunks(BT, true);
  const int nseg_h = segments_for(a.din, cap);
  if (nseg_h * 2 > kWaves) return hipErrorInvalidValue;
  const int per = (nch + nseg_h * kWave - 1) / (nseg_h * kWave);
  if (per <= 1) return launch_seg<BT, 1>(a, m, nseg_h, s, ev);
  if constexpr (BT <= 2) {
    if (per <= 2) return launch_seg<BT, 2>(a, m, nseg_h, s, ev);
    if (per <= 3) return launch_seg<BT, 3>(a, m, nseg_h, s, ev);
  }
  if constexpr (BT == 1) {
    if (per <= 4) return launch_seg<BT, 4>(a, m, nseg_h, s, ev);
    return launch_seg<BT, 6>(a, m, nseg_h, s, ev);
  }
  return hipErrorInvalidValue;
}

}  // namespace

int mlp_fused_blocks(int inter) { return inter < kNumCu ? inter : kNumCu; }
int mlp_fused_u8(int inter) {
  const int G = mlp_fused_blocks(inter);
  return ((inter + G - 1) / G + 7) / 8 * 8;
}

hipError_t launch_mlp_fused(const GemvArgs& a, const MlpFusedArgs& m, hipStream_t s, KernelEvents ev_slice,
                            KernelEvents ev_reduce) {
  if (m.nblk != mlp_fused_blocks(a.rows) || m.u8 != mlp_fused_u8(a.rows) || m.hidden != a.din) return hipErrorInvalidValue;
  hipError_t e;
  if (a.batch >= 4 && segments_for(a.din, max_chunks(4, true)) * 2 <= kWaves)
    e = launch_bt<4>(a, m, s, ev_slice);
  else if (a.batch >= 2 && segments_for(a.din, max_chunks(2, true)) * 2 <= kWaves)
    e = launch_bt<2>(a, m, s, ev_slice);
  else
    e = launch_bt<1>(a, m, s, ev_slice);
  if (e != hipSuccess) return e;
  dim3 grid((m.hidden + kRedOut - 1) / kRedOut, a.batch);
  return ext_launch(mlp_reduce_kernel, grid, dim3(256), 0, s, ev_reduce, m, (const float*)a.in_f32, m.y);
}

hipError_t launch_pack_down_slices(const uint16_t* w_down, uint16_t* dst, int hidden, int inter, hipStream_t s) {
  const int G = mlp_fused_blocks(inter), u8 = mlp_fused_u8(inter);
  hipLaunchKernelGGL(pack_down_slices_kernel, dim3(G, hidden), dim3(64), 0, s, w_down, dst, hidden, inter, G, u8);
  return hipGetLastError();
}

}  // namespace fasttps
