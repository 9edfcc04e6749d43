// Host-side launchers of the gfx950 kernels (internal to libfasttps).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fasttps {

constexpr int kMaxBatch = 64;

// Optional start/stop events of one launch (null: plain launch). They are
// set from the dispatch packet itself, so timing adds nothing to the stream.
struct KernelEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};

template <typename... Params, typename... Args>
inline hipError_t ext_launch(void (*kernel)(Params...), dim3 grid, dim3 block, size_t lds, hipStream_t s,
                             KernelEvents ev, Args... args) {
  static_assert(sizeof...(Params) == sizeof...(Args), "argument count");
  void* argv[] = {static_cast<void*>(&args)...};
  return hipExtLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, argv, lds, s, ev.start, ev.stop,
                            0);
}

struct PosArray {
  int32_t p[kMaxBatch];
};

// y[b, r] = sum_c W[r, c] * act[b, c] over `rows` rows of a bf16 [rows, din]
// matrix ([rows, 2 din] for the gate/up pairs).
struct GemvArgs {
  const uint16_t* w;       // [rows, din] bf16 (gate/up: [rows, 2 din], row k = [gate k | up k])
  int rows, din, batch;
  const uint16_t* x_bf16;  // QKV: token x [batch, din]; O proj: residual x [batch, rows]
  const uint16_t* gamma;   // QKV, gate/up: RMSNorm gain [din]
  const float* in_f32;     // O proj, down: activation [batch, din]; gate/up: h1 [batch, din] (fp32)
  float* out;              // QKV, O proj, gate/up: [batch, rows] fp32
  const float* res_f32;    // down: residual h1 [batch, rows] fp32
  uint16_t* out_bf16;      // down: y [batch, rows] bf16
  float eps;
  int ld;                  // elements per stored row of w (0: din, or 2 din for gate/up)
  float* dbg_act;          // test hook, null in normal steps: QKV and gate/up write the
                           // normalized activation (RMSNorm1(x) resp. RMSNorm2(h1)) [batch, din]
};

// RMSNorm1(x) followed by the fused QKV projection (fp32 out, before RoPE).
hipError_t launch_rmsnorm_qkv(const GemvArgs& a, hipStream_t s, KernelEvents ev = {});
// h1 = x + W_o o  (fp32 out).
hipError_t launch_oproj_residual(const GemvArgs& a, hipStream_t s, KernelEvents ev = {});
// y = bf16(h1 + W_down a)  (din = K up to 32768).
hipError_t launch_down_residual(const GemvArgs& a, hipStream_t s, KernelEvents ev = {});
// a = SiLU(W_gate h2) * (W_up h2), h2 = RMSNorm2(h1), over the interlaced
// W_gu with tiles of one row (rows = K).
hipError_t launch_gate_up(const GemvArgs& a, hipStream_t s, KernelEvents ev = {});
// out = W act (fp32 in and out), rows of `ld` elements (the op-by-op baseline).
hipError_t launch_gemv_plain(const GemvArgs& a, hipStream_t s, KernelEvents ev = {});

// The O projection of one sequence with the merge of the attention's split
// partials in its prologue (gemv.hip), in place of a separate combine kernel:
// every block merges all heads' splits into o in LDS (the log-sum-exp merge
// of Alg. 3's softmax over the splits), then streams its rows of W_o as
// launch_oproj_residual does; block 0 also stores o.
struct MergeArgs {
  const float* part;  // [H, nsplit_cap, d + kPartLead] (m, l, -, -, o) of each split, sequence 0
  float* o;           // [H d] fp32
  int nsplit, nsplit_cap, n_heads, head_dim;
};
constexpr int kMergeMaxSplits = 16;
constexpr int kMergeMaxElems = 4096;  // H d
bool oproj_merge_supported(int n_heads, int head_dim, int nsplit, int rows);
// a: the O projection's GemvArgs (batch 1; in_f32 unused)
hipError_t launch_oproj_merge(const GemvArgs& a, const MergeArgs& m, hipStream_t s, KernelEvents ev = {});

// The fused MLP (mlp_fused.hip): gate/up + siLu_Mul of a slice of units per
// block with h^sm kept in LDS, the slice's down-projection partial of y, and
// a fixed-order sum of the partials with the residual.
struct MlpFusedArgs {
  const uint16_t* w_down_slices;  // [nblk][hidden][u8] bf16 (launch_pack_down_slices)
  float* part;                    // [nblk][batch][hidden] fp32 partials of W_down a
  uint16_t* y;                    // [batch][hidden] bf16 output
  int nblk, u8, hidden, batch;
};
int mlp_fused_blocks(int inter);  // blocks (slices) of the fused MLP
int mlp_fused_u8(int inter);      // units per slice, rounded up to a multiple of 8
// a: the gate/up GemvArgs (w = interlaced W_gu, in_f32 = h1, gamma = RMSNorm2 gain)
hipError_t launch_mlp_fused(const GemvArgs& a, const MlpFusedArgs& m, hipStream_t s, KernelEvents ev_slice = {},
                            KernelEvents ev_reduce = {});
hipError_t launch_pack_down_slices(const uint16_t* w_down, uint16_t* dst, int hidden, int inter, hipStream_t s);

// Batched projections on the matrix cores: out = W act over weights packed
// in MFMA tiles (16 rows x 32 inputs, 1 KB, in operand order) and
// activations split into two bf16 levels (see mfma_proj.hip).
struct MfmaArgs {
  const uint16_t* w;        // tiled weights [ns][kt][64 lanes][8] bf16
  int ns, kt, nt;           // stripes, k-tiles (32 inputs), k-tiles per wave (ceil(kt / 16))
  int rh;                   // rows per stripe, even, <= 16 (gate/up: rh / 2 units)
  int sch;                  // stripes per LDS chunk of partial sums (set by the launcher)
  int rows, din, batch;     // real output rows (gate/up: units K), real inputs, sequences
  int nbtc;                 // batch tiles (8 sequences) of the a_in buffer
  const uint16_t* x_bf16;   // QKV: token x [batch, din]; O proj: residual x [batch, rows]
  const uint16_t* gamma;    // QKV: RMSNorm1 gain [din]; O proj: RMSNorm2 gain [rows]
  const uint16_t* a_in;     // O proj, gate/up, down: the operand [kt][nbtc][64][8] bf16
  float* out;               // QKV: q|k|v [batch, rows]; O proj: h1; gate/up: a (fp32)
  uint16_t* a_out;          // O proj, gate/up: the next projection's operand
  int a_out_nbtc;           // its batch tiles
  float* ssq_out;           // O proj: per-stripe sums of h1^2 [ns][batch]
  const float* ssq_in;      // gate/up: those sums [ns_in][batch]
  int ns_in;
  const float* res_f32;     // down: residual h1 [batch, rows]
  uint16_t* out_bf16;       // down: y [batch, rows] bf16
  float eps;
  // split inputs (O, gate/up, down): scratch for the parts' fp32 partial sums
  // and the row groups' tickets (zero between launches; every launch leaves
  // them zero), with their sizes (mfma_split_need); null: no split
  float* kpart;
  unsigned* tickets;
  size_t kpart_cap, tickets_cap;
  int ks, ktq, kstride;     // set by the launcher: parts, k-tiles per part, floats per block of kpart
};
// the split scratch a projection needs at up to `batch` sequences (mode 0
// QKV, 1 O, 2 gate/up, 3 down; ns stripes of rh rows and kt k-tiles)
void mfma_split_need(int mode, int ns, int kt, int rh, int batch, size_t* kpart_floats, size_t* tickets);
hipError_t launch_mfma_qkv(const MfmaArgs& a, hipStream_t s, KernelEvents ev = {});
hipError_t launch_mfma_oproj(const MfmaArgs& a, hipStream_t s, KernelEvents ev = {});
hipError_t launch_mfma_gate_up(const MfmaArgs& a, hipStream_t s, KernelEvents ev = {});
hipError_t launch_mfma_down(const MfmaArgs& a, hipStream_t s, KernelEvents ev = {});
// the MFMA-tiled copy of a row-major [rows, din] matrix with row stride ld,
// in stripes of rh rows; with `up` set, stripes of rh / 2 rows of src (gate)
// and the rh / 2 matching rows of up
hipError_t launch_tile_weights(const uint16_t* src, const uint16_t* up, int rows, int din, int ld, int ns, int kt,
                               int rh, uint16_t* dst, hipStream_t s);

// A split's partial softmax state in the attention's scratch: m, l, two unused
// floats, then o[d], so that o starts on a 16-byte boundary.
constexpr int kPartLead = 4;

struct AttnArgs {
  const float* qkv;        // [batch, (H + 2 H_kv) d] fp32, before RoPE
  const double* rope_cos;  // [N_max, d/2]
  const double* rope_sin;  // [N_max, d/2]
  void* k_cache;           // [B, H_kv, N_max, d], bf16 or 8-bit codes
  void* v_cache;
  float* part;             // [batch, H, nsplit_cap, d + kPartLead] split partials (m, l, -, -, o)
  float* o;                // [batch, H d] fp32
  uint16_t* o_operand;     // if set: o split for the MFMA O projection [kt][o_nbtc][64][8]
  int o_nbtc;
  int batch, n_heads, n_kv_heads, head_dim, max_seq;
  int nsplit, nsplit_cap;     // splits per (sequence, KV head): split s takes tiles s, s + nsplit, ...
  float scale;             // 1/sqrt(d)
  int p_bf16;              // accuracy study: softmax weights rounded to bf16 before PV
  int kv_format;           // kKvBf16, kKvFp8 or kKvInt8
  PosArray pos;
  PosArray order;          // grid z -> sequence: the longest first, so the shortest blocks go last
  float* dbg_qk;           // test hook, null in normal steps: q and k after RoPE (fp32)
                           // [batch, (H + H_kv) d], q heads first
};
// cache element formats (the values of the ABI's FASTTPS_KV_* constants)
constexpr int kKvBf16 = 0, kKvFp8 = 1, kKvInt8 = 2;
constexpr int kMaxKvHeads = 128;  // n_heads * head_dim <= 8192, head_dim >= 64
// the per-KV-head scales of an 8-bit cache, passed by value
struct KvScales {
  float k[kMaxKvHeads];
  float v[kMaxKvHeads];
};
// per split: RoPE, append, partial softmax state (m, l, o)
hipError_t launch_attention(const AttnArgs& a, hipStream_t s, KernelEvents ev = {});
// the same over an 8-bit cache (a.kv_format kKvFp8 or kKvInt8)
hipError_t launch_attention_kv8(const AttnArgs& a, const KvScales& sc, hipStream_t s, KernelEvents ev = {});
// combine the split partials into o
hipError_t launch_attention_combine(const AttnArgs& a, hipStream_t s, KernelEvents ev = {});

// The whole step of one sequence as one persistent kernel (fused_layer.hip):
// the four projections' arguments (fp32 outputs and inputs in the layer's
// scratch), the attention's, and the phase hand-over state.
struct FusedArgs {
  GemvArgs qkv, oproj, gateup, down;
  AttnArgs attn;
  unsigned* flags;   // [5][256] per-block phase flags (epochs)
  unsigned* epoch;   // the last completed launch's epoch (device)
  int* err;          // count of bounded waits that ran out (device)
  int attn_items;    // nsplit * n_kv_heads
  int stage_floats;  // max(H d, D, K): the LDS stage of a projection's input
};
// The launch shapes of the step's projections (GEMV chunks per lane, segments
// per half row, rows in flight) and the attention's head dimension and group.
struct FusedShape {
  struct Gemv {
    int maxch, nseg_h, nbuf;
    bool operator==(const Gemv& o) const { return maxch == o.maxch && nseg_h == o.nseg_h && nbuf == o.nbuf; }
  };
  int head_dim, group;
  Gemv q, o, gu, down;
};
bool fused_layer_supported(const FusedShape& sh);
int fused_layer_max_splits();  // attention splits per KV head the kernel merges
int fused_layer_grid();        // its blocks (one (KV head, split) item each at most)
hipError_t launch_fused_layer(const FusedArgs& f, const FusedShape& sh, hipStream_t s, KernelEvents ev = {});
// the chunks per lane, segments per half row and ring depth the separate
// GEMV kernels use for one sequence (their blocks have 8 or 16 waves; the
// fused kernel's rows are dealt to its 16-wave blocks with the same shape)
FusedShape::Gemv gemv_shape_b1(int din, bool gate_up);

// The op-by-op baseline (Alg. 1 + Alg. 2, every intermediate through HBM).
struct UnfusedArgs {
  const uint16_t* x;                       // [B, D] bf16
  const uint16_t *attn_norm, *mlp_norm;    // [D]
  const uint16_t *w_qkv, *w_o, *w_gu, *w_down;  // packed weights
  uint16_t *k_cache, *v_cache;             // [B, H_kv, N_max, d], slot pos_b written
  uint16_t* y;                             // [B, D] bf16
  const double *rope_cos, *rope_sin;       // [N_max, d/2]
  float *h, *q, *k, *v, *q_rope, *k_rope, *q_t, *k_t, *v_t;  // fp32 intermediates
  uint16_t *kcat, *vcat;                   // the concatenated caches [B, H_kv, N_max, d]
  float *S, *P;                            // [B, H, N_max]
  float* pv_part;                          // [B, H, pv_cap, d]
  float *O, *attn_out, *h1, *h2, *g, *sg, *up, *hp, *mlp_out;
  int batch, hidden, n_heads, n_kv_heads, head_dim, inter, max_seq, maxn, pv_cap;
  float scale, eps;
  PosArray pos;
};
hipError_t launch_unfused(const UnfusedArgs& u, hipStream_t s);
int unfused_pv_splits(int max_seq);

// packing (cold path)
hipError_t launch_interlace_gate_up(const uint16_t* gate, const uint16_t* up, uint16_t* dst, int inter,
                                    int hidden, int tk, hipStream_t s);

}  // namespace fasttps
