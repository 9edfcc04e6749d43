// The op-by-op decode layer (gfx950): the paper's standard implementation,
// Alg. 1 (RoPE, Transpose, Concat, QK^T, Softmax, PV) and Alg. 2 (gate, SiLU,
// up, elementwise mul, down), each operator a kernel of its own whose inputs
// and outputs go through HBM, with the Concat that rebuilds the cache in a
// new buffer (the reloading GKVC removes, Section 3.1.1). It is the baseline
// the fused layer is measured against; the projections use the same GEMV
// kernel as the fused path, so the comparison isolates the fusion.
#include "common.h"
#include "kernels.h"

#include <math.h>

namespace fasttps {

namespace {

constexpr int kThreads = 256;

// h[b] = x[b] / sqrt(mean(x[b]^2) + eps) * gamma; x bf16 or fp32 (one block of
// 1024 threads per row; the row is read once into registers)
constexpr int kNormThreads = 1024;
constexpr int kNormPer = 8;  // hidden <= 8192, the layer's limit

template <bool BF16_IN>
__global__ __launch_bounds__(kNormThreads) void rmsnorm_kernel(const void* __restrict__ x,
                                                               const uint16_t* __restrict__ gamma,
                                                               float* __restrict__ h, int D, float eps) {
  __shared__ float red[kNormThreads / kWave];
  const int b = blockIdx.x;
  float xv[kNormPer];
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < kNormPer; ++k) {
    const int i = threadIdx.x + k * kNormThreads;
    const int ic = min(i, D - 1);
    const float v = BF16_IN ? bf16_to_f32(static_cast<const uint16_t*>(x)[(size_t)b * D + ic])
                            : static_cast<const float*>(x)[(size_t)b * D + ic];
    xv[k] = i < D ? v : 0.f;
    ss = fmaf(xv[k], xv[k], ss);
  }
  const float tot = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(tot / (float)D + eps);
#pragma unroll
  for (int k = 0; k < kNormPer; ++k) {
    const int i = threadIdx.x + k * kNormThreads;
    if (i < D) h[(size_t)b * D + i] = xv[k] * inv * bf16_to_f32(gamma[i]);
  }
}

// RoPE of `nh` heads of d values per sequence (rotate-half, fp64 cos/sin row of
// the sequence's position), fp32 in and out; one block per (head, sequence).
__global__ __launch_bounds__(kThreads) void rope_kernel(const float* __restrict__ in, float* __restrict__ out, int nh,
                                                        int d, const double* __restrict__ cs,
                                                        const double* __restrict__ sn, PosArray pos) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int half = d / 2;
  const double* c = cs + (size_t)pos.p[b] * half;
  const double* s = sn + (size_t)pos.p[b] * half;
  const float* x = in + ((size_t)b * nh + h) * d;
  float* y = out + ((size_t)b * nh + h) * d;
  for (int j = threadIdx.x; j < half; j += kThreads) {
    const double a0 = x[j], a1 = x[j + half];
    y[j] = (float)(a0 * c[j] - a1 * s[j]);
    y[j + half] = (float)(a1 * c[j] + a0 * s[j]);
  }
}

// [B, N = 1, H, d] -> [B, H, N = 1, d]: with one token the layouts coincide, and
// the operator is the copy the standard pipeline makes.
__global__ __launch_bounds__(kThreads) void transpose_kernel(const float* __restrict__ in, float* __restrict__ out,
                                                             int n) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i < n) out[i] = in[i];
}

// Concat: cat[b, g, 0 .. pos_b] = [cache[b, g, 0 .. pos_b), bf16(new[b, g])] in a
// new buffer, and the new entry also into the caller's cache slot pos_b (the
// in-place state the next step reads). One thread per 16-byte chunk.
__global__ __launch_bounds__(kThreads) void concat_kernel(const uint16_t* cache, const float* __restrict__ knew,
                                                          uint16_t* __restrict__ cat, uint16_t* cache_out,
                                                          int Hkv, int nmax, int d, PosArray pos) {
  const int g = blockIdx.y, b = blockIdx.z;
  const int c8 = d / 8;
  const int q = blockIdx.x * kThreads + threadIdx.x;  // chunk over [nmax, c8]
  const int n = q / c8, c = q % c8;
  const int P = pos.p[b];
  if (n > P) return;
  const size_t row = ((size_t)b * Hkv + g) * nmax + n;
  v4u val;
  if (n < P) {
    val = reinterpret_cast<const v4u*>(cache + row * d)[c];
  } else {
    const float* k = knew + ((size_t)b * Hkv + g) * d + 8 * c;
    val = v4u{(uint32_t)f32_to_bf16(k[0]) | ((uint32_t)f32_to_bf16(k[1]) << 16),
              (uint32_t)f32_to_bf16(k[2]) | ((uint32_t)f32_to_bf16(k[3]) << 16),
              (uint32_t)f32_to_bf16(k[4]) | ((uint32_t)f32_to_bf16(k[5]) << 16),
              (uint32_t)f32_to_bf16(k[6]) | ((uint32_t)f32_to_bf16(k[7]) << 16)};
    reinterpret_cast<v4u*>(cache_out + row * d)[c] = val;
  }
  reinterpret_cast<v4u*>(cat + row * d)[c] = val;
}

// S[b, h, j] = q[b, h] . K[b, g, j] * scale for j <= pos_b (g = h / G); four
// lanes per position, 64 positions per block.
template <int D>
__global__ __launch_bounds__(kThreads) void qk_kernel(const float* __restrict__ q, const uint16_t* __restrict__ kcat,
                                                      float* __restrict__ S, int H, int Hkv, int nmax, float scale,
                                                      PosArray pos) {
  constexpr int SEG = D / 4;
  const int h = blockIdx.y, b = blockIdx.z;
  const int g = h / (H / Hkv);
  const int j = blockIdx.x * 64 + (threadIdx.x >> 2), seg = threadIdx.x & 3;
  const int P = pos.p[b];
  const int jc = min(j, P);  // lanes past the end compute a valid row and do not store
  const v4u* kr = reinterpret_cast<const v4u*>(kcat + (((size_t)b * Hkv + g) * nmax + jc) * D + seg * SEG);
  const float* qh = q + ((size_t)b * H + h) * D + seg * SEG;
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < SEG / 8; ++c) {
    float kf[8];
    unpack8(kr[c], kf);
#pragma unroll
    for (int e = 0; e < 8; ++e) s = fmaf(qh[8 * c + e], kf[e], s);
  }
  s = quad_sum(s) * scale;
  if (j <= P && seg == 0) S[((size_t)b * H + h) * nmax + j] = s;
}

// P[b, h, 0 .. pos_b] = softmax(S[b, h, 0 .. pos_b]); one block per (head, sequence).
__global__ __launch_bounds__(1024) void softmax_kernel(const float* __restrict__ S, float* __restrict__ Pm, int H,
                                                       int nmax, PosArray pos) {
  __shared__ float red[1024 / kWave];
  const int h = blockIdx.x, b = blockIdx.y;
  const int n = pos.p[b] + 1;
  const float* s = S + ((size_t)b * H + h) * nmax;
  float* p = Pm + ((size_t)b * H + h) * nmax;
  float m = -INFINITY;
  for (int i = threadIdx.x; i < n; i += blockDim.x) m = fmaxf(m, s[i]);
  m = wave_max(m);
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = m;
  __syncthreads();
  float M = red[0];
  for (int w = 1; w < (int)blockDim.x / kWave; ++w) M = fmaxf(M, red[w]);
  __syncthreads();
  float l = 0.f;
  for (int i = threadIdx.x; i < n; i += blockDim.x) l += expf(s[i] - M);
  const float L = block_sum(l, red);
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = expf(s[i] - M) / L;
}

// Partial O over 256 positions: part[b, h, split, :] = sum_j P[b, h, j] V[b, g, j, :]
// (four lanes per position, a quarter of d each; 64 positions at a time).
constexpr int kPvSplit = 256;

template <int D>
__global__ __launch_bounds__(kThreads) void pv_kernel(const float* __restrict__ Pm, const uint16_t* __restrict__ vcat,
                                                      float* __restrict__ part, int H, int Hkv, int nmax,
                                                      int nsplit_cap, PosArray pos) {
  constexpr int SEG = D / 4;
  __shared__ float red[kThreads / 16][D];
  const int s = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int g = h / (H / Hkv);
  const int P = pos.p[b];
  const int j0 = threadIdx.x >> 2, seg = threadIdx.x & 3;
  float o[SEG];
#pragma unroll
  for (int e = 0; e < SEG; ++e) o[e] = 0.f;
  const float* p = Pm + ((size_t)b * H + h) * nmax;
  for (int j = s * kPvSplit + j0; j < min((s + 1) * kPvSplit, P + 1); j += 64) {
    const float pj = p[j];
    const v4u* vr = reinterpret_cast<const v4u*>(vcat + (((size_t)b * Hkv + g) * nmax + j) * D + seg * SEG);
#pragma unroll
    for (int c = 0; c < SEG / 8; ++c) {
      float vf[8];
      unpack8(vr[c], vf);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[8 * c + e] = fmaf(pj, vf[e], o[8 * c + e]);
    }
  }
  // the 4 positions of each 16-lane row, then the 16 rows
#pragma unroll
  for (int e = 0; e < SEG; ++e) o[e] = row_stride4_sum(o[e]);
  const int row = threadIdx.x >> 4;
  if ((threadIdx.x & 15) < 4)
#pragma unroll
    for (int e = 0; e < SEG; ++e) red[row][seg * SEG + e] = o[e];
  __syncthreads();
  for (int e = threadIdx.x; e < D; e += kThreads) {
    float t = 0.f;
    for (int r = 0; r < kThreads / 16; ++r) t += red[r][e];
    part[(((size_t)b * H + h) * nsplit_cap + s) * D + e] = t;
  }
}

// O[b, h, :] = sum over splits of the partials
__global__ __launch_bounds__(kThreads) void pv_reduce_kernel(const float* __restrict__ part, float* __restrict__ O,
                                                             int H, int D, int nsplit_cap, PosArray pos) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int nsplit = (pos.p[b] + 1 + kPvSplit - 1) / kPvSplit;
  for (int e = threadIdx.x; e < D; e += kThreads) {
    float t = 0.f;
    for (int s = 0; s < nsplit; ++s) t += part[(((size_t)b * H + h) * nsplit_cap + s) * D + e];
    O[((size_t)b * H + h) * D + e] = t;
  }
}

// out = x + y (x bf16 or fp32; out fp32, or bf16 rounded)
template <bool X_BF16, bool OUT_BF16>
__global__ __launch_bounds__(kThreads) void add_kernel(const void* __restrict__ x, const float* __restrict__ y,
                                                       void* __restrict__ out, int n) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= n) return;
  const float xv = X_BF16 ? bf16_to_f32(static_cast<const uint16_t*>(x)[i]) : static_cast<const float*>(x)[i];
  const float v = xv + y[i];
  if (OUT_BF16) static_cast<uint16_t*>(out)[i] = f32_to_bf16(v);
  else static_cast<float*>(out)[i] = v;
}

__global__ __launch_bounds__(kThreads) void silu_kernel(const float* __restrict__ g, float* __restrict__ s, int n) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i < n) s[i] = g[i] / (1.0f + expf(-g[i]));
}

__global__ __launch_bounds__(kThreads) void mul_kernel(const float* __restrict__ a, const float* __restrict__ b,
                                                       float* __restrict__ c, int n) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i < n) c[i] = a[i] * b[i];
}

inline dim3 grid1(int n) { return dim3((n + kThreads - 1) / kThreads); }

template <int D>
hipError_t launch_attn_ops(const UnfusedArgs& u, hipStream_t s) {
  const int B = u.batch, H = u.n_heads, Hkv = u.n_kv_heads;
  // QK^T over the concatenated cache
  hipLaunchKernelGGL(qk_kernel<D>, dim3((u.maxn + 63) / 64, H, B), dim3(kThreads), 0, s, u.q_t, u.kcat, u.S, H, Hkv,
                     u.max_seq, u.scale, u.pos);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(softmax_kernel, dim3(H, B), dim3(1024), 0, s, u.S, u.P, H, u.max_seq, u.pos);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(pv_kernel<D>, dim3((u.maxn + kPvSplit - 1) / kPvSplit, H, B), dim3(kThreads), 0, s, u.P, u.vcat,
                     u.pv_part, H, Hkv, u.max_seq, u.pv_cap, u.pos);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(pv_reduce_kernel, dim3(H, B), dim3(kThreads), 0, s, u.pv_part, u.O, H, D, u.pv_cap, u.pos);
  return hipGetLastError();
}

}  // namespace

int unfused_pv_splits(int max_seq) { return (max_seq + kPvSplit - 1) / kPvSplit; }

hipError_t launch_unfused(const UnfusedArgs& u, hipStream_t s) {
  const int B = u.batch, D = u.hidden, H = u.n_heads, Hkv = u.n_kv_heads, d = u.head_dim, K = u.inter;
  const int qd = H * d, kvd = Hkv * d;
  hipError_t e;
  auto gemv = [&](const uint16_t* w, int rows, int din, int ld, const float* act, float* out) {
    GemvArgs g{};
    g.w = w;
    g.rows = rows;
    g.din = din;
    g.batch = B;
    g.in_f32 = act;
    g.out = out;
    g.ld = ld;
    return launch_gemv_plain(g, s);
  };
  // ---- attention block (Alg. 1) ------------------------------------------
  hipLaunchKernelGGL(rmsnorm_kernel<true>, dim3(B), dim3(kNormThreads), 0, s, u.x, u.attn_norm, u.h, D, u.eps);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = gemv(u.w_qkv, qd, D, 0, u.h, u.q)) != hipSuccess) return e;
  if ((e = gemv(u.w_qkv + (size_t)qd * D, kvd, D, 0, u.h, u.k)) != hipSuccess) return e;
  if ((e = gemv(u.w_qkv + (size_t)(qd + kvd) * D, kvd, D, 0, u.h, u.v)) != hipSuccess) return e;
  // Step 1: RoPE on Q and K
  hipLaunchKernelGGL(rope_kernel, dim3(H, B), dim3(kThreads), 0, s, u.q, u.q_rope, H, d, u.rope_cos, u.rope_sin, u.pos);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(rope_kernel, dim3(Hkv, B), dim3(kThreads), 0, s, u.k, u.k_rope, Hkv, d, u.rope_cos, u.rope_sin,
                     u.pos);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // Step 2: Transpose
  hipLaunchKernelGGL(transpose_kernel, grid1(B * qd), dim3(kThreads), 0, s, u.q_rope, u.q_t, B * qd);
  hipLaunchKernelGGL(transpose_kernel, grid1(B * kvd), dim3(kThreads), 0, s, u.k_rope, u.k_t, B * kvd);
  hipLaunchKernelGGL(transpose_kernel, grid1(B * kvd), dim3(kThreads), 0, s, u.v, u.v_t, B * kvd);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // Step 3: Concat of K and of V with their caches, into new buffers
  const dim3 cgrid((u.max_seq * (d / 8) + kThreads - 1) / kThreads, Hkv, B);
  hipLaunchKernelGGL(concat_kernel, cgrid, dim3(kThreads), 0, s, u.k_cache, u.k_t, u.kcat, u.k_cache, Hkv, u.max_seq,
                     d, u.pos);
  hipLaunchKernelGGL(concat_kernel, cgrid, dim3(kThreads), 0, s, u.v_cache, u.v_t, u.vcat, u.v_cache, Hkv, u.max_seq,
                     d, u.pos);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // Steps 4-6: QK^T, Softmax, PV
  switch (d) {
    case 64: e = launch_attn_ops<64>(u, s); break;
    case 96: e = launch_attn_ops<96>(u, s); break;
    case 128: e = launch_attn_ops<128>(u, s); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  // O projection, residual
  if ((e = gemv(u.w_o, D, qd, 0, u.O, u.attn_out)) != hipSuccess) return e;
  hipLaunchKernelGGL((add_kernel<true, false>), grid1(B * D), dim3(kThreads), 0, s, u.x, u.attn_out, u.h1, B * D);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // ---- MLP block (Alg. 2) ------------------------------------------------
  hipLaunchKernelGGL(rmsnorm_kernel<false>, dim3(B), dim3(kNormThreads), 0, s, u.h1, u.mlp_norm, u.h2, D, u.eps);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // Step 1: gate projection (the even rows of the interlaced W_gu), Step 2: SiLU
  if ((e = gemv(u.w_gu, K, D, 2 * D, u.h2, u.g)) != hipSuccess) return e;
  hipLaunchKernelGGL(silu_kernel, grid1(B * K), dim3(kThreads), 0, s, u.g, u.sg, B * K);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // Step 3: up projection (the odd rows), Step 4: elementwise mul
  if ((e = gemv(u.w_gu + D, K, D, 2 * D, u.h2, u.up)) != hipSuccess) return e;
  hipLaunchKernelGGL(mul_kernel, grid1(B * K), dim3(kThreads), 0, s, u.sg, u.up, u.hp, B * K);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // Step 5: down projection, then the residual and the bf16 output
  if ((e = gemv(u.w_down, D, K, 0, u.hp, u.mlp_out)) != hipSuccess) return e;
  hipLaunchKernelGGL((add_kernel<false, true>), grid1(B * D), dim3(kThreads), 0, s, u.h1, u.mlp_out, u.y, B * D);
  return hipGetLastError();
}

}  // namespace fasttps
