// Weight packing kernels (cold path, run once per layer at pack time).
#include "common.h"
#include "kernels.h"

namespace fasttps {

namespace {

// Interlaced W_gu (Section 3.2 item 1, Alg. 4): destination rows come in
// tiles of 2*tk: tk rows of W_gate, then the tk matching rows of W_up. The
// last tile holds 2*(K - i*tk) rows when tk does not divide K.
__global__ __launch_bounds__(256) void interlace_kernel(const uint16_t* __restrict__ gate,
                                                        const uint16_t* __restrict__ up,
                                                        uint16_t* __restrict__ dst, int inter, int hidden,
                                                        int tk) {
  const int r = blockIdx.x;  // destination row in [0, 2K)
  const int tile = r / (2 * tk);
  const int within = r % (2 * tk);
  const int k0 = tile * tk;
  const int tkb = min(tk, inter - k0);
  const bool is_up = within >= tkb;
  const int src_row = k0 + (is_up ? within - tkb : within);
  const uint4* src = reinterpret_cast<const uint4*>((is_up ? up : gate) + (size_t)src_row * hidden);
  uint4* d = reinterpret_cast<uint4*>(dst + (size_t)r * hidden);
  for (int c = threadIdx.x; c < hidden / 8; c += blockDim.x) d[c] = src[c];
}

// dst[c][r] = src[r][c] for a [rows, cols] bf16 matrix, through 32x32 LDS tiles.
__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t* __restrict__ src,
                                                        uint16_t* __restrict__ dst, int rows, int cols) {
  __shared__ uint16_t tile[32][33];
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
  for (int i = ty; i < 32; i += 8) {
    const int r = r0 + i, c = c0 + tx;
    if (r < rows && c < cols) tile[i][tx] = src[(size_t)r * cols + c];
  }
  __syncthreads();
  for (int i = ty; i < 32; i += 8) {
    const int c = c0 + i, r = r0 + tx;
    if (r < rows && c < cols) dst[(size_t)c * rows + r] = tile[tx][i];
  }
}

}  // namespace

hipError_t launch_interlace_gate_up(const uint16_t* gate, const uint16_t* up, uint16_t* dst, int inter,
                                    int hidden, int tk, hipStream_t s) {
  hipLaunchKernelGGL(interlace_kernel, dim3(2 * inter), dim3(256), 0, s, gate, up, dst, inter, hidden, tk);
  return hipGetLastError();
}

hipError_t launch_transpose_bf16(const uint16_t* src, uint16_t* dst, int rows, int cols, hipStream_t s) {
  dim3 grid((cols + 31) / 32, (rows + 31) / 32);
  hipLaunchKernelGGL(transpose_kernel, grid, dim3(256), 0, s, src, dst, rows, cols);
  return hipGetLastError();
}

}  // namespace fasttps
