// Device helpers shared by the gfx950 kernels of the FastTPS decode layer.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace fasttps {

constexpr int kWave = 64;

// a compile-time flag passed to a generic lambda (the body of a loop's last
// round and of the rounds before it)
template <bool B>
struct BoolTag {
  static constexpr bool value = B;
};

// 16 bytes as a native vector: copies of it are plain vector moves, so
// staging arrays of it stay in registers (HIP's uint4 struct is copied with
// memcpy, which can pin such arrays to scratch memory).
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// A load of data the step reads once (weights, cached K/V), with the
// non-temporal cache policy (global_load ... nt). On MI355X a 4 GiB stream of
// 16-byte nt loads reads 7.1-7.2 TB/s against 6.3-6.4 TB/s for plain loads at
// every launch shape tried (256-16384 blocks, 4 or 8 loads in flight per lane).
template <typename T>
__device__ __forceinline__ T ld_stream(const T* p) {
  return __builtin_nontemporal_load(p);
}

// ---- data handed between blocks of one launch ----------------------------
// The L2 caches are per XCD and not coherent with each other. Data another
// block reads in the same launch is stored and loaded with the accesses of
// relaxed agent-scope atomics (global_store / global_load sc1), which bypass
// the non-coherent L2, so no L2 write-back or invalidate is needed; the
// writer waits for its stores (wait_vm) before it signals.
__device__ __forceinline__ float ld_c(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_c(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned ld_cu(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_cu(unsigned* p, unsigned v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// The log-sum-exp merge's factor of a partial softmax state with running
// maximum m against the merged maximum M (zero for an empty state).
__device__ __forceinline__ float merge_factor(float m, float M) {
  return (m == -INFINITY) ? 0.f : __expf(m - M);
}

// wait for this wave's outstanding memory operations, stores included
// (s_waitcnt vmcnt(0); expcnt and lgkmcnt left free)
__device__ __forceinline__ void wait_vm() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// ---- bfloat16 <-> float -------------------------------------------------
// bf16 is the upper half of a binary32, so widening is a shift.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// float -> bf16, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x0040u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// double -> bf16 with a single rounding (nearest even): first to float with
// round-to-odd (truncate, then set the last bit if anything was dropped),
// which keeps the information a second nearest-even rounding needs because
// float carries 16 more significand bits than bf16.
__device__ __forceinline__ uint16_t f64_to_bf16(double x) {
  float t = __double2float_rz(x);
  uint32_t u = __float_as_uint(t);
  if ((double)t != x && x == x) u |= 1u;
  return f32_to_bf16(__uint_as_float(u));
}

// Eight bf16 (one 16-byte load) dotted with eight floats.
__device__ __forceinline__ float dot8(const uint4 w, const float* h) {
  float s = bf16_lo(w.x) * h[0];
  s = fmaf(bf16_hi(w.x), h[1], s);
  s = fmaf(bf16_lo(w.y), h[2], s);
  s = fmaf(bf16_hi(w.y), h[3], s);
  s = fmaf(bf16_lo(w.z), h[4], s);
  s = fmaf(bf16_hi(w.z), h[5], s);
  s = fmaf(bf16_lo(w.w), h[6], s);
  s = fmaf(bf16_hi(w.w), h[7], s);
  return s;
}

__device__ __forceinline__ float fma8(const uint4 w, const float* h, float acc) {
  acc = fmaf(bf16_lo(w.x), h[0], acc);
  acc = fmaf(bf16_hi(w.x), h[1], acc);
  acc = fmaf(bf16_lo(w.y), h[2], acc);
  acc = fmaf(bf16_hi(w.y), h[3], acc);
  acc = fmaf(bf16_lo(w.z), h[4], acc);
  acc = fmaf(bf16_hi(w.z), h[5], acc);
  acc = fmaf(bf16_lo(w.w), h[6], acc);
  acc = fmaf(bf16_hi(w.w), h[7], acc);
  return acc;
}

__device__ __forceinline__ void unpack8(const uint4 w, float* f) {
  f[0] = bf16_lo(w.x); f[1] = bf16_hi(w.x);
  f[2] = bf16_lo(w.y); f[3] = bf16_hi(w.y);
  f[4] = bf16_lo(w.z); f[5] = bf16_hi(w.z);
  f[6] = bf16_lo(w.w); f[7] = bf16_hi(w.w);
}

__device__ __forceinline__ void unpack8(const v4u w, float* f) {
  f[0] = bf16_lo(w.x); f[1] = bf16_hi(w.x);
  f[2] = bf16_lo(w.y); f[3] = bf16_hi(w.y);
  f[4] = bf16_lo(w.z); f[5] = bf16_hi(w.z);
  f[6] = bf16_lo(w.w); f[7] = bf16_hi(w.w);
}

// ---- data-parallel-primitive (DPP) lane moves ---------------------------
// Full-rate VALU moves between lanes of a quad (4 lanes) or a row (16
// lanes); __shfl_xor goes through the LDS crossbar (ds_bpermute) instead.
constexpr int kDppQuadXor1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;  // quad_perm [2,3,0,1]
constexpr int kDppRowRor4 = 0x124;  // rotate right by 4 within each row of 16
constexpr int kDppRowRor8 = 0x128;  // rotate right by 8 within each row of 16

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}

// 16 bytes of the neighbouring lane (lane ^ 1)
__device__ __forceinline__ v4u dpp_swap_pair(v4u v) {
  return v4u{(unsigned)__builtin_amdgcn_mov_dpp((int)v.x, kDppQuadXor1, 0xF, 0xF, false),
             (unsigned)__builtin_amdgcn_mov_dpp((int)v.y, kDppQuadXor1, 0xF, 0xF, false),
             (unsigned)__builtin_amdgcn_mov_dpp((int)v.z, kDppQuadXor1, 0xF, 0xF, false),
             (unsigned)__builtin_amdgcn_mov_dpp((int)v.w, kDppQuadXor1, 0xF, 0xF, false)};
}

// Sum over the 4 lanes of a quad; every lane gets the result.
__device__ __forceinline__ float quad_sum(float v) {
  v += dpp_mov<kDppQuadXor1>(v);
  return v + dpp_mov<kDppQuadXor2>(v);
}

// Sum / max over the lanes of a 16-lane row that share lane % 4; every lane
// gets the result for its residue.
__device__ __forceinline__ float row_stride4_sum(float v) {
  v += dpp_mov<kDppRowRor4>(v);
  return v + dpp_mov<kDppRowRor8>(v);
}
__device__ __forceinline__ float row_stride4_max(float v) {
  v = fmaxf(v, dpp_mov<kDppRowRor4>(v));
  return fmaxf(v, dpp_mov<kDppRowRor8>(v));
}

// ---- wavefront reductions (64 lanes) ------------------------------------
// Quad and row steps by DPP, then the row totals are chained with the
// row_bcast15 / row_bcast31 moves (rows 1 and 3 add the total of the row
// before; rows 2 and 3 add lane 31), which leaves the wave total in lane 63;
// a readlane hands it to every lane. The order of the additions is fixed.
constexpr int kDppRowBcast15 = 0x142;
constexpr int kDppRowBcast31 = 0x143;

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_upd(float old, float v) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(v), CTRL, ROW_MASK, 0xF, false));
}

__device__ __forceinline__ float wave_sum(float v) {
  v = row_stride4_sum(quad_sum(v));           // every lane: its row's total
  v += dpp_upd<kDppRowBcast15, 0xA>(0.f, v);  // rows 1, 3: + previous row
  v += dpp_upd<kDppRowBcast31, 0xC>(0.f, v);  // rows 2, 3: + rows 0..1
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_mov<kDppQuadXor1>(v));
  v = fmaxf(v, dpp_mov<kDppQuadXor2>(v));
  v = row_stride4_max(v);
  v = fmaxf(v, dpp_upd<kDppRowBcast15, 0xA>(v, v));
  v = fmaxf(v, dpp_upd<kDppRowBcast31, 0xC>(v, v));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// Sum of v over the whole block; every thread gets the total. `red` must
// hold blockDim.x / 64 floats.
__device__ __forceinline__ float block_sum(float v, float* red) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float t = 0.f;
  const int nw = blockDim.x / kWave;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

}  // namespace fasttps
