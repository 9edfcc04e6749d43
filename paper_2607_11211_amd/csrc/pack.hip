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

}  // namespace

hipError_t launch_interlace_gate_up(const uint16_t* gate, const uint16_t* up, uint16_t* dst, int inter,
                                    int hidden, int tk, hipStream_t s) {
  hipLaunchKernelGGL(interlace_kernel, dim3(2 * inter), dim3(256), 0, s, gate, up, dst, inter, hidden, tk);
  return hipGetLastError();
}

}  // namespace fasttps
