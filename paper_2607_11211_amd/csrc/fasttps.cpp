// C ABI of the FastTPS decode layer: validation, ownership, launch sequence.
#include "fasttps.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <unordered_set>
#include <vector>

#include "kernels.h"

using namespace fasttps;

namespace {

constexpr uint64_t kLayerMagic = 0x4641535454505331ull;    // "FASTTPS1"
constexpr uint64_t kWeightsMagic = 0x4641535454505357ull;  // "FASTTPSW"
constexpr uint64_t kDeadMagic = 0xDEADDEADDEADDEADull;
// attention blocks per step (256 CUs): 2 per CU (each lane with two tiles in
// flight for one or two query heads per KV head, one for groups of four);
// four times as many, shorter splits when the batch's positions are ragged.
// Measured on MI355X: Phi-3 16-sequence ragged batch 101 -> 94 us and GQA
// 4 x 32768 115 -> 103 us against 768 blocks throughout; then 512 blocks with
// two tiles in flight against 768 with one: Phi-3 layer at KV 4096 61.7 ->
// 61.2 us per step, 16-sequence ragged batch attention 87.9 -> 86.3 us; and
// for the GQA layer 512 blocks against 256 (one per CU): 193-195 -> 188-189
// us per step (384 and 1024 slower).
constexpr int kTargetAttnBlocks = 512;
// One sequence: about one block per CU, so that the split partials the O
// projection's blocks merge stay small (8 splits of the Phi-3 layer's 32
// heads, 128 KB). Measured on MI355X (Phi-3 layer at KV 4096, HIP graph):
// the attention is as fast at 256 blocks as at 512 (11.2-11.5 us); with 128
// blocks it takes 12.8 us.
constexpr int kTargetAttnBlocksOne = 256;
constexpr int kRaggedAttnFactor = 4;
constexpr int kAttnTile = 64;
constexpr int kMaxSplits = 256;

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(FASTTPS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

int round_up(int v, int m) { return (v + m - 1) / m * m; }
int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Shapes of the MFMA-tiled matrices: stripes of rh output rows (gate/up:
// rh / 2 units, i.e. rh / 2 gate and rh / 2 up rows) by k-tiles of 32 inputs.
struct TileDims {
  int ns, kt, rh;
  size_t elems() const { return (size_t)ns * kt * 32 * rh; }
};
struct LayerTiles {
  TileDims qkv, o, gu, down;
};
// The stripe height (16, 12 or 8 rows) that gives the most loaded of the
// kMfmaBlocks blocks the fewest rows (units of `per_row` rows for gate/up),
// the tallest on ties: 9216 rows go in 768 stripes of 12 (3 per block), 3072
// in 256 of 12, 4096 in 256 of 16.
constexpr int kMfmaBlocks = 256;
TileDims pick_tiles(int rows, int din, int per_row) {
  TileDims best{0, ceil_div(din, 32), 0};
  long best_load = 0;
  for (int rh : {16, 12, 8}) {
    const int units = rh / per_row;
    const int ns = ceil_div(rows, units);
    const int g = std::min(ns, kMfmaBlocks);
    const long load = (long)ceil_div(ns, g) * units;
    if (best.rh == 0 || load < best_load) {
      best = {ns, ceil_div(din, 32), rh};
      best_load = load;
    }
  }
  return best;
}
LayerTiles layer_tiles(const fasttps_config& c) {
  const int D = c.hidden, K = c.intermediate, q = c.n_heads * c.head_dim;
  const int rows_qkv = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim;
  return {pick_tiles(rows_qkv, D, 1), pick_tiles(D, q, 1), pick_tiles(K, D, 2), pick_tiles(D, K, 1)};
}
// the fused kernel: phases with a flag per block, and its grid
constexpr int kFusedPhases = 5;
constexpr int kFusedBlocks = 256;

// the MFMA path is taken from this batch size up (FASTTPS_GEMM_AUTO)
constexpr int kMfmaMinBatch = 2;
constexpr int kMfmaWaves = 16;  // waves per block of the MFMA kernels (they split the k-tiles)

// Interlaced W_gu (Section 3.2 item 1, Alg. 4) in tiles of one row: packed
// row 2k is W_gate row k, row 2k + 1 is W_up row k, so the gate/up pair of an
// intermediate unit is one contiguous 2D-value row for the projection kernel.
constexpr int kInterlaceTile = 1;

// test-hook buffers a step wrote (fasttps_layer::dbg_written)
constexpr int kDbgQk = 1, kDbgNorm = 2;

// The allocation-free step's scratch (fasttps_decode_step_noalloc): one
// statically sized array per device, reached through the address
// hipGetSymbolAddress gives for each device (the array's name in host code
// is a stand-in, not a device address). Looked up once per device by
// fasttps_layer_create, with that device current.
constexpr size_t kStaticScratchBytes = size_t(8) << 20;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {

// The device address of this device's static scratch array (dev current).
hipError_t static_scratch_lookup(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev]) return hipSuccess;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  g_scratch_ptr[dev] = p;
  return hipSuccess;
}

void* static_scratch(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  return g_scratch_ptr[dev];
}

}  // namespace

struct fasttps_layer {
  uint64_t magic;
  fasttps_config cfg;
  int device;
  int nsplit_cap;
  int p_bf16 = 0;  // accuracy study switch (fasttps_set_attention_p_bf16)
  int debug = 0;   // test hook switch (fasttps_set_debug)
  // what the last step wrote to the test-hook buffers: kDbgQk (q, k after
  // RoPE), kDbgNorm (the two normalized activations; vector path only)
  int dbg_written = 0;
  void* arena;
  double* rope_cos;
  double* rope_sin;
  float* qkv;
  float* attn_part;
  float* attn_o;
  float* h1;
  float* mlp_a;
  // test-hook outputs: q | k after RoPE [B, (H + H_kv) d], RMSNorm1(x) and
  // RMSNorm2(h1) [B, D]
  float* dbg_qk;
  float* dbg_h;
  float* dbg_h2;
  // operands of the MFMA projections (layers with max_batch > 1): o, h1 * gamma2
  // and SiLU(g) * u split into bf16 levels in lane order, and RMSNorm2's
  // per-stripe sums of squares
  uint16_t* op_o = nullptr;
  uint16_t* op_gu = nullptr;
  uint16_t* op_down = nullptr;
  float* ssq_h1 = nullptr;
  int nbtc = 0;        // batch tiles of the operand buffers
  float* split_part = nullptr;    // the split projections' partial sums
  unsigned* split_tickets = nullptr;  // and their row groups' tickets (zero between steps)
  size_t split_part_cap = 0, split_tickets_cap = 0;
  int gemm_path = FASTTPS_GEMM_AUTO;
  // the MLP as one kernel with h^sm on chip (fasttps_set_mlp_path): its
  // partial sums of y [slices][max_batch][D], allocated when first selected
  int mlp_path = FASTTPS_MLP_SPLIT;
  int weight_layout = FASTTPS_WEIGHTS_ROWS_AND_TILES;  // how later packs store the projections
  float* mlp_part = nullptr;
  bool mlp_a_written = false;  // the last step stored h^sm (FASTTPS_DBG_MLP_A)
  // the fused kernel's phase hand-over: per-block phase flags, the epoch of
  // the last completed launch, the count of bounded waits that ran out
  unsigned* fused_flags = nullptr;
  unsigned* fused_epoch = nullptr;
  int* fused_err = nullptr;
  // the op-by-op baseline's scratch (fasttps_unfused_enable)
  void* uf_arena = nullptr;
  UnfusedArgs uf{};
  // per-kernel timing (measurement hook)
  std::vector<hipEvent_t> prof_events;  // [cap][kernel][start, stop]
  std::vector<uint8_t> prof_used;       // [cap][kernel]: launched with its events
  int prof_cap = 0;
  int prof_n = 0;
};

struct fasttps_weights {
  uint64_t magic;
  fasttps_config cfg;
  void* arena;
  uint16_t* w_qkv;
  uint16_t* w_o;
  uint16_t* w_gu;
  uint16_t* w_down;
  uint16_t* attn_norm;
  uint16_t* mlp_norm;
  // MFMA tiles (16 rows x 32 inputs in operand order), packed for layers with
  // max_batch > 1; null otherwise
  uint16_t* t_qkv = nullptr;
  uint16_t* t_o = nullptr;
  uint16_t* t_gu = nullptr;
  uint16_t* t_down = nullptr;
  // W_down in the fused MLP's slices [slices][D][u8], packed when the layer
  // handle used for packing had the fused MLP selected; null otherwise
  uint16_t* w_down_slices = nullptr;
};

namespace {

int validate_config(const fasttps_config* c) {
  if (!c) return fail(FASTTPS_ERR_INVALID_ARG, "config is null");
  if (c->hidden <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 || c->intermediate <= 0 ||
      c->max_batch <= 0 || c->max_seq <= 0)
    return fail(FASTTPS_ERR_INVALID_ARG, "config sizes must be positive");
  if (c->max_batch > kMaxBatch) return fail(FASTTPS_ERR_INVALID_ARG, "max_batch %d > %d", c->max_batch, kMaxBatch);
  if (!(std::isfinite(c->rope_base) && c->rope_base > 1.0f))
    return fail(FASTTPS_ERR_INVALID_ARG, "rope_base must be finite and > 1");
  if (!(std::isfinite(c->rms_eps) && c->rms_eps > 0.0f))
    return fail(FASTTPS_ERR_INVALID_ARG, "rms_eps must be finite and > 0");
  if (c->hidden % 8 != 0 || c->hidden > 8192)
    return fail(FASTTPS_ERR_UNSUPPORTED, "hidden %d: need a multiple of 8 up to 8192", c->hidden);
  if (c->head_dim != 64 && c->head_dim != 96 && c->head_dim != 128)
    return fail(FASTTPS_ERR_UNSUPPORTED, "head_dim %d: supported 64, 96, 128", c->head_dim);
  if (c->n_heads % c->n_kv_heads != 0) return fail(FASTTPS_ERR_UNSUPPORTED, "n_heads %% n_kv_heads != 0");
  const int group = c->n_heads / c->n_kv_heads;
  if (group != 1 && group != 2 && group != 4)
    return fail(FASTTPS_ERR_UNSUPPORTED, "n_heads / n_kv_heads = %d: supported 1, 2, 4", group);
  if ((long)c->n_heads * c->head_dim > 8192)
    return fail(FASTTPS_ERR_UNSUPPORTED, "n_heads * head_dim > 8192");
  if (c->intermediate % 8 != 0 || c->intermediate > 32768)
    return fail(FASTTPS_ERR_UNSUPPORTED, "intermediate %d: need a multiple of 8 up to 32768", c->intermediate);
  if ((long)c->max_seq * c->head_dim * c->n_kv_heads * c->max_batch > (1L << 40))
    return fail(FASTTPS_ERR_UNSUPPORTED, "cache too large");
  return FASTTPS_OK;
}

bool same_shape(const fasttps_config& a, const fasttps_config& b) {
  return a.hidden == b.hidden && a.n_heads == b.n_heads && a.n_kv_heads == b.n_kv_heads &&
         a.head_dim == b.head_dim && a.intermediate == b.intermediate;
}

// Live handles: a handle is dereferenced only after it is found here, so a
// stale or foreign pointer is reported instead of read.
std::mutex g_handles_mu;
std::unordered_set<const void*> g_layers, g_weights;

void track(std::unordered_set<const void*>& set, const void* p, bool add) {
  std::lock_guard<std::mutex> lk(g_handles_mu);
  if (add)
    set.insert(p);
  else
    set.erase(p);
}

bool live(const std::unordered_set<const void*>& set, const void* p) {
  std::lock_guard<std::mutex> lk(g_handles_mu);
  return p && set.count(p) != 0;
}

bool layer_ok(const fasttps_layer* l) { return live(g_layers, l) && l->magic == kLayerMagic; }
bool weights_ok(const fasttps_weights* w) { return live(g_weights, w) && w->magic == kWeightsMagic; }

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

void release_events(fasttps_layer* l) {
  for (hipEvent_t e : l->prof_events) (void)hipEventDestroy(e);
  l->prof_events.clear();
  l->prof_used.clear();
  l->prof_cap = 0;
  l->prof_n = 0;
}

}  // namespace

extern "C" {

const char* fasttps_status_string(int status) {
  switch (status) {
    case FASTTPS_OK: return "ok";
    case FASTTPS_ERR_INVALID_ARG: return "invalid argument";
    case FASTTPS_ERR_UNSUPPORTED: return "unsupported shape";
    case FASTTPS_ERR_ALIGNMENT: return "pointer not 16-byte aligned";
    case FASTTPS_ERR_CACHE_FULL: return "cache full or bad position";
    case FASTTPS_ERR_OOM: return "device allocation failed";
    case FASTTPS_ERR_HIP: return "HIP runtime error";
    case FASTTPS_ERR_BAD_HANDLE: return "bad handle";
    default: return "unknown status";
  }
}

const char* fasttps_last_error(void) { return g_last_error.c_str(); }

int fasttps_layer_create(const fasttps_config* cfg, fasttps_layer** out) {
  g_last_error.clear();
  if (!out) return fail(FASTTPS_ERR_INVALID_ARG, "out is null");
  *out = nullptr;
  int st = validate_config(cfg);
  if (st) return st;
  const fasttps_config c = *cfg;
  const int d = c.head_dim, half = d / 2;
  const int B = c.max_batch;
  const int nsplit_cap = std::min(
      {kMaxSplits, ceil_div(kRaggedAttnFactor * kTargetAttnBlocks, c.n_kv_heads), ceil_div(c.max_seq, kAttnTile)});
  const size_t qkv_rows = (size_t)(c.n_heads + 2 * c.n_kv_heads) * d;

  // RoPE table in double precision: angle(n, j) = n * base^(-2j/d)
  std::vector<double> cs((size_t)c.max_seq * half), sn((size_t)c.max_seq * half);
  for (int j = 0; j < half; ++j) {
    const double inv_freq = std::pow((double)c.rope_base, -2.0 * (double)j / (double)d);
    for (int n = 0; n < c.max_seq; ++n) {
      const double th = (double)n * inv_freq;
      cs[(size_t)n * half + j] = std::cos(th);
      sn[(size_t)n * half + j] = std::sin(th);
    }
  }

  const bool mfma = B > 1;
  const int nbtc = 2 * ceil_div(B, 16);
  const LayerTiles lt = layer_tiles(c);
  // the split projections run one after another: one scratch serves them all
  size_t split_floats = 0, split_tickets = 0;
  if (mfma) {
    const TileDims* tds[3] = {&lt.o, &lt.gu, &lt.down};
    for (int i = 0; i < 3; ++i) {
      size_t f = 0, t = 0;
      mfma_split_need(i + 1, tds[i]->ns, tds[i]->kt, tds[i]->rh, B, &f, &t);
      split_floats = std::max(split_floats, f);
      split_tickets = std::max(split_tickets, t);
    }
  }
  size_t sizes[17] = {
      cs.size() * sizeof(double),
      sn.size() * sizeof(double),
      (size_t)B * qkv_rows * sizeof(float),
      (size_t)B * c.n_heads * nsplit_cap * (d + kPartLead) * sizeof(float),
      (size_t)B * c.n_heads * d * sizeof(float),
      (size_t)B * c.hidden * sizeof(float),
      (size_t)B * c.intermediate * sizeof(float),
      mfma ? (size_t)lt.o.kt * nbtc * 512 * sizeof(uint16_t) : 0,
      mfma ? (size_t)lt.gu.kt * nbtc * 512 * sizeof(uint16_t) : 0,
      mfma ? (size_t)lt.down.kt * nbtc * 512 * sizeof(uint16_t) : 0,
      mfma ? (size_t)lt.o.ns * B * sizeof(float) : 0,
      (size_t)kFusedPhases * kFusedBlocks * sizeof(unsigned) + 2 * sizeof(unsigned),
      (size_t)B * (c.n_heads + c.n_kv_heads) * d * sizeof(float),
      (size_t)B * c.hidden * sizeof(float),
      (size_t)B * c.hidden * sizeof(float),
      split_floats * sizeof(float),
      split_tickets * sizeof(unsigned),
  };
  size_t total = 0, offs[17];
  for (int i = 0; i < 17; ++i) {
    offs[i] = total;
    total += align256(sizes[i]);
  }

  fasttps_layer* l = new (std::nothrow) fasttps_layer();
  if (!l) return fail(FASTTPS_ERR_OOM, "host allocation failed");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    delete l;
    return hip_fail(e, "hipGetDevice");
  }
  if ((e = static_scratch_lookup(dev)) != hipSuccess) {
    delete l;
    return hip_fail(e, "hipGetSymbolAddress of the static scratch");
  }
  void* arena = nullptr;
  e = hipMalloc(&arena, total);
  if (e != hipSuccess) {
    delete l;
    (void)hipGetLastError();
    return fail(FASTTPS_ERR_OOM, "hipMalloc(%zu): %s", total, hipGetErrorString(e));
  }
  char* base = static_cast<char*>(arena);
  l->magic = kLayerMagic;
  l->cfg = c;
  l->device = dev;
  l->nsplit_cap = nsplit_cap;
  l->arena = arena;
  l->rope_cos = reinterpret_cast<double*>(base + offs[0]);
  l->rope_sin = reinterpret_cast<double*>(base + offs[1]);
  l->qkv = reinterpret_cast<float*>(base + offs[2]);
  l->attn_part = reinterpret_cast<float*>(base + offs[3]);
  l->attn_o = reinterpret_cast<float*>(base + offs[4]);
  l->h1 = reinterpret_cast<float*>(base + offs[5]);
  l->mlp_a = reinterpret_cast<float*>(base + offs[6]);
  if (mfma) {
    l->op_o = reinterpret_cast<uint16_t*>(base + offs[7]);
    l->op_gu = reinterpret_cast<uint16_t*>(base + offs[8]);
    l->op_down = reinterpret_cast<uint16_t*>(base + offs[9]);
    l->ssq_h1 = reinterpret_cast<float*>(base + offs[10]);
    l->nbtc = nbtc;
    if (split_floats && split_tickets) {
      l->split_part = reinterpret_cast<float*>(base + offs[15]);
      l->split_tickets = reinterpret_cast<unsigned*>(base + offs[16]);
      l->split_part_cap = split_floats;
      l->split_tickets_cap = split_tickets;
    }
  }
  l->fused_flags = reinterpret_cast<unsigned*>(base + offs[11]);
  l->fused_epoch = l->fused_flags + kFusedPhases * kFusedBlocks;
  l->fused_err = reinterpret_cast<int*>(l->fused_epoch + 1);
  l->dbg_qk = reinterpret_cast<float*>(base + offs[12]);
  l->dbg_h = reinterpret_cast<float*>(base + offs[13]);
  l->dbg_h2 = reinterpret_cast<float*>(base + offs[14]);

  // the operand buffers start at zero: their padding (inputs past the
  // matrix's last column) must stay zero, since the padded weights are zero
  // and 0 * NaN is not
  if ((e = hipMemcpy(l->rope_cos, cs.data(), sizes[0], hipMemcpyHostToDevice)) != hipSuccess ||
      (e = hipMemcpy(l->rope_sin, sn.data(), sizes[1], hipMemcpyHostToDevice)) != hipSuccess ||
      (e = hipMemset(base + offs[2], 0, total - offs[2])) != hipSuccess ||
      (e = hipDeviceSynchronize()) != hipSuccess) {
    (void)hipFree(arena);
    l->magic = kDeadMagic;
    delete l;
    return hip_fail(e, "layer setup");
  }
  track(g_layers, l, true);
  *out = l;
  return FASTTPS_OK;
}

int fasttps_layer_destroy(fasttps_layer* l) {
  g_last_error.clear();
  if (!layer_ok(l)) return fail(FASTTPS_ERR_BAD_HANDLE, "layer handle is null or already destroyed");
  track(g_layers, l, false);
  release_events(l);
  l->magic = kDeadMagic;
  hipError_t e = hipFree(l->arena);
  if (l->mlp_part) {
    const hipError_t e2 = hipFree(l->mlp_part);
    if (e == hipSuccess) e = e2;
  }
  if (l->uf_arena) {
    const hipError_t e2 = hipFree(l->uf_arena);
    if (e == hipSuccess) e = e2;
  }
  delete l;
  if (e != hipSuccess) return hip_fail(e, "hipFree");
  return FASTTPS_OK;
}

const char* fasttps_kernel_name(int32_t k) {
  static const char* names[FASTTPS_NUM_KERNELS] = {"rmsnorm_qkv",    "attention",   "attn_combine", "oproj_residual",
                                                   "mlp_gate_up", "mlp_down", "fused_layer"};
  return (k >= 0 && k < FASTTPS_NUM_KERNELS) ? names[k] : "";
}

int fasttps_profile_begin(fasttps_layer* l, int32_t max_steps) {
  g_last_error.clear();
  if (!layer_ok(l)) return fail(FASTTPS_ERR_BAD_HANDLE, "bad layer handle");
  if (max_steps < 1 || max_steps > (1 << 16)) return fail(FASTTPS_ERR_INVALID_ARG, "max_steps out of range");
  release_events(l);
  l->prof_events.resize((size_t)max_steps * FASTTPS_NUM_KERNELS * 2, nullptr);
  l->prof_used.assign((size_t)max_steps * FASTTPS_NUM_KERNELS, 0);
  for (auto& ev : l->prof_events) {
    hipError_t e = hipEventCreate(&ev);
    if (e != hipSuccess) {
      ev = nullptr;
      release_events(l);
      return hip_fail(e, "hipEventCreate");
    }
  }
  l->prof_cap = max_steps;
  l->prof_n = 0;
  return FASTTPS_OK;
}

int fasttps_profile_end(fasttps_layer* l, float* ms, int32_t max_steps, int32_t* n_steps) {
  g_last_error.clear();
  if (!layer_ok(l)) return fail(FASTTPS_ERR_BAD_HANDLE, "bad layer handle");
  if (!ms || !n_steps) return fail(FASTTPS_ERR_INVALID_ARG, "null output");
  const int n = std::min(l->prof_n, (int)max_steps);
  *n_steps = n;
  hipError_t e = hipSuccess;
  // the last launched kernel of the last recorded step
  if (l->prof_n > 0) {
    const size_t st = (size_t)(l->prof_n - 1) * FASTTPS_NUM_KERNELS;
    int kl = FASTTPS_NUM_KERNELS - 1;
    while (kl > 0 && !l->prof_used[st + kl]) --kl;
    e = hipEventSynchronize(l->prof_events[(st + kl) * 2 + 1]);
  }
  for (int i = 0; i < n && e == hipSuccess; ++i)
    for (int k = 0; k < FASTTPS_NUM_KERNELS && e == hipSuccess; ++k) {
      const size_t j = (size_t)i * FASTTPS_NUM_KERNELS + k;
      ms[j] = 0.f;
      if (l->prof_used[j]) e = hipEventElapsedTime(&ms[j], l->prof_events[2 * j], l->prof_events[2 * j + 1]);
    }
  release_events(l);
  if (e != hipSuccess) return hip_fail(e, "kernel timing");
  return FASTTPS_OK;
}

int fasttps_weights_pack(fasttps_layer* l, const fasttps_weights_desc* w, void* stream, fasttps_weights** out) {
  g_last_error.clear();
  if (!out) return fail(FASTTPS_ERR_INVALID_ARG, "out is null");
  *out = nullptr;
  if (!layer_ok(l)) return fail(FASTTPS_ERR_BAD_HANDLE, "bad layer handle");
  if (!w) return fail(FASTTPS_ERR_INVALID_ARG, "weights descriptor is null");
  const void* ptrs[9] = {w->attn_norm, w->w_q, w->w_k, w->w_v, w->w_o, w->mlp_norm, w->w_gate, w->w_up, w->w_down};
  for (int i = 0; i < 9; ++i) {
    if (!ptrs[i]) return fail(FASTTPS_ERR_INVALID_ARG, "weight pointer %d is null", i);
    if (!aligned16(ptrs[i])) return fail(FASTTPS_ERR_ALIGNMENT, "weight pointer %d is not 16-byte aligned", i);
  }
  const fasttps_config& c = l->cfg;
  const size_t D = c.hidden, K = c.intermediate, d = c.head_dim;
  const size_t q = (size_t)c.n_heads * d, kv = (size_t)c.n_kv_heads * d;
  const size_t n_qkv = (q + 2 * kv) * D, n_o = D * q, n_gu = 2 * K * D, n_d = K * D;
  const bool tiled = c.max_batch > 1;
  const bool rows = !tiled || l->weight_layout == FASTTPS_WEIGHTS_ROWS_AND_TILES;  // row-major copies
  const LayerTiles lt = layer_tiles(c);
  const bool slices = l->mlp_path == FASTTPS_MLP_FUSED;
  if (slices && !rows)
    return fail(FASTTPS_ERR_INVALID_ARG, "the fused MLP needs row-major weights (layout FASTTPS_WEIGHTS_TILES set)");
  const size_t n_sl = (size_t)mlp_fused_blocks((int)K) * D * mlp_fused_u8((int)K);
  size_t offs[11], sizes[11] = {rows ? n_qkv * 2 : 0, rows ? n_o * 2 : 0, rows ? n_gu * 2 : 0, rows ? n_d * 2 : 0,
                                D * 2, D * 2,
                                tiled ? lt.qkv.elems() * 2 : 0, tiled ? lt.o.elems() * 2 : 0,
                                tiled ? lt.gu.elems() * 2 : 0, tiled ? lt.down.elems() * 2 : 0,
                                slices ? n_sl * 2 : 0};
  size_t total = 0;
  for (int i = 0; i < 11; ++i) {
    offs[i] = total;
    total += align256(sizes[i]);
  }
  fasttps_weights* pw = new (std::nothrow) fasttps_weights();
  if (!pw) return fail(FASTTPS_ERR_OOM, "host allocation failed");
  void* arena = nullptr;
  hipError_t e = hipMalloc(&arena, total);
  if (e != hipSuccess) {
    delete pw;
    (void)hipGetLastError();
    return fail(FASTTPS_ERR_OOM, "hipMalloc(%zu): %s", total, hipGetErrorString(e));
  }
  char* base = static_cast<char*>(arena);
  pw->magic = kWeightsMagic;
  pw->cfg = c;
  pw->arena = arena;
  if (rows) {
    pw->w_qkv = reinterpret_cast<uint16_t*>(base + offs[0]);
    pw->w_o = reinterpret_cast<uint16_t*>(base + offs[1]);
    pw->w_gu = reinterpret_cast<uint16_t*>(base + offs[2]);
    pw->w_down = reinterpret_cast<uint16_t*>(base + offs[3]);
  }
  pw->attn_norm = reinterpret_cast<uint16_t*>(base + offs[4]);
  pw->mlp_norm = reinterpret_cast<uint16_t*>(base + offs[5]);
  if (tiled) {
    pw->t_qkv = reinterpret_cast<uint16_t*>(base + offs[6]);
    pw->t_o = reinterpret_cast<uint16_t*>(base + offs[7]);
    pw->t_gu = reinterpret_cast<uint16_t*>(base + offs[8]);
    pw->t_down = reinterpret_cast<uint16_t*>(base + offs[9]);
  }
  if (slices) pw->w_down_slices = reinterpret_cast<uint16_t*>(base + offs[10]);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const auto* g = static_cast<const uint16_t*>(w->w_gate);
  const auto* u = static_cast<const uint16_t*>(w->w_up);
  // the tile order only: the tiles come from the caller's matrices, W_q|W_k|W_v
  // through a temporary row-major copy (freed before returning)
  void* qkv_tmp = nullptr;
  if (!rows && (e = hipMalloc(&qkv_tmp, n_qkv * 2)) != hipSuccess) {
    (void)hipGetLastError();
    (void)hipFree(arena);
    pw->magic = kDeadMagic;
    delete pw;
    return fail(FASTTPS_ERR_OOM, "hipMalloc(%zu): %s", n_qkv * 2, hipGetErrorString(e));
  }
  uint16_t* qkv_rows = rows ? pw->w_qkv : static_cast<uint16_t*>(qkv_tmp);
  const uint16_t* o_rows = rows ? pw->w_o : static_cast<const uint16_t*>(w->w_o);
  const uint16_t* down_rows = rows ? pw->w_down : static_cast<const uint16_t*>(w->w_down);
  if ((e = hipMemcpyAsync(qkv_rows, w->w_q, q * D * 2, hipMemcpyDeviceToDevice, s)) != hipSuccess ||
      (e = hipMemcpyAsync(qkv_rows + q * D, w->w_k, kv * D * 2, hipMemcpyDeviceToDevice, s)) != hipSuccess ||
      (e = hipMemcpyAsync(qkv_rows + (q + kv) * D, w->w_v, kv * D * 2, hipMemcpyDeviceToDevice, s)) != hipSuccess ||
      (rows && (e = hipMemcpyAsync(pw->w_o, w->w_o, n_o * 2, hipMemcpyDeviceToDevice, s)) != hipSuccess) ||
      (e = hipMemcpyAsync(pw->attn_norm, w->attn_norm, D * 2, hipMemcpyDeviceToDevice, s)) != hipSuccess ||
      (e = hipMemcpyAsync(pw->mlp_norm, w->mlp_norm, D * 2, hipMemcpyDeviceToDevice, s)) != hipSuccess ||
      (rows && (e = launch_interlace_gate_up(g, u, pw->w_gu, (int)K, (int)D, kInterlaceTile, s)) != hipSuccess) ||
      (rows && (e = hipMemcpyAsync(pw->w_down, w->w_down, n_d * 2, hipMemcpyDeviceToDevice, s)) != hipSuccess) ||
      (slices && (e = launch_pack_down_slices(pw->w_down, pw->w_down_slices, (int)D, (int)K, s)) != hipSuccess) ||
      (tiled && ((e = launch_tile_weights(qkv_rows, nullptr, (int)(q + 2 * kv), (int)D, (int)D, lt.qkv.ns,
                                          lt.qkv.kt, lt.qkv.rh, pw->t_qkv, s)) != hipSuccess ||
                 (e = launch_tile_weights(o_rows, nullptr, (int)D, (int)q, (int)q, lt.o.ns, lt.o.kt, lt.o.rh,
                                          pw->t_o, s)) != hipSuccess ||
                 (e = launch_tile_weights(g, u, (int)K, (int)D, (int)D, lt.gu.ns, lt.gu.kt, lt.gu.rh, pw->t_gu, s)) !=
                     hipSuccess ||
                 (e = launch_tile_weights(down_rows, nullptr, (int)D, (int)K, (int)K, lt.down.ns, lt.down.kt,
                                          lt.down.rh, pw->t_down, s)) != hipSuccess)) ||
      (e = hipStreamSynchronize(s)) != hipSuccess) {
    (void)hipStreamSynchronize(s);
    if (qkv_tmp) (void)hipFree(qkv_tmp);
    (void)hipFree(arena);
    pw->magic = kDeadMagic;
    delete pw;
    return hip_fail(e, "weight packing");
  }
  if (qkv_tmp && (e = hipFree(qkv_tmp)) != hipSuccess) {
    (void)hipFree(arena);
    pw->magic = kDeadMagic;
    delete pw;
    return hip_fail(e, "hipFree of the packing copy");
  }
  track(g_weights, pw, true);
  *out = pw;
  return FASTTPS_OK;
}

int fasttps_weights_free(fasttps_weights* w) {
  g_last_error.clear();
  if (!weights_ok(w)) return fail(FASTTPS_ERR_BAD_HANDLE, "weights handle is null or already freed");
  track(g_weights, w, false);
  w->magic = kDeadMagic;
  hipError_t e = hipFree(w->arena);
  delete w;
  if (e != hipSuccess) return hip_fail(e, "hipFree");
  return FASTTPS_OK;
}

namespace {

// The argument checks of a step against a layer config (no handle, no HIP
// call); on success *maxp is the largest position of the batch.
int check_args(const fasttps_config& c, const void* x, const int32_t* pos, int32_t batch, const void* k_cache,
               const void* v_cache, const void* y, int* maxp, size_t cache_elem_bytes) {
  if (!x || !pos || !k_cache || !v_cache || !y) return fail(FASTTPS_ERR_INVALID_ARG, "null pointer argument");
  if (batch < 1 || batch > c.max_batch)
    return fail(FASTTPS_ERR_INVALID_ARG, "batch %d outside [1, %d]", batch, c.max_batch);
  if (!aligned16(x) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(y))
    return fail(FASTTPS_ERR_ALIGNMENT, "tensor pointers must be 16-byte aligned");
  int mp = 0;
  for (int b = 0; b < batch; ++b) {
    if (pos[b] < 0 || pos[b] >= c.max_seq)
      return fail(FASTTPS_ERR_CACHE_FULL, "pos[%d] = %d outside [0, %d)", b, pos[b], c.max_seq);
    mp = std::max(mp, pos[b]);
  }
  const size_t D = c.hidden, d = c.head_dim;
  const size_t act_bytes = (size_t)batch * D * 2;
  const size_t cache_bytes = (size_t)batch * c.n_kv_heads * c.max_seq * d * cache_elem_bytes;
  if (overlaps(y, act_bytes, x, act_bytes) || overlaps(y, act_bytes, k_cache, cache_bytes) ||
      overlaps(y, act_bytes, v_cache, cache_bytes))
    return fail(FASTTPS_ERR_INVALID_ARG, "y overlaps x or a cache");
  if (overlaps(k_cache, cache_bytes, v_cache, cache_bytes))
    return fail(FASTTPS_ERR_INVALID_ARG, "k_cache and v_cache overlap");
  *maxp = mp;
  return FASTTPS_OK;
}

// The checks shared by the step entry points: the handles, then the
// arguments. Makes no HIP call.
int check_step(fasttps_layer* l, const fasttps_weights* w, const void* x, const int32_t* pos, int32_t batch,
               void* k_cache, void* v_cache, void* y, int* maxp, size_t cache_elem_bytes = 2) {
  if (!layer_ok(l)) return fail(FASTTPS_ERR_BAD_HANDLE, "bad layer handle");
  if (!weights_ok(w)) return fail(FASTTPS_ERR_BAD_HANDLE, "bad weights handle");
  if (!same_shape(l->cfg, w->cfg))
    return fail(FASTTPS_ERR_BAD_HANDLE, "weights were packed for another layer shape");
  return check_args(l->cfg, x, pos, batch, k_cache, v_cache, y, maxp, cache_elem_bytes);
}

}  // namespace

int fasttps_validate_step(const fasttps_config* cfg, const void* x, const int32_t* pos, int32_t batch,
                          const void* k_cache, const void* v_cache, const void* y, int32_t cache_elem_bytes) {
  g_last_error.clear();
  int st = validate_config(cfg);
  if (st) return st;
  if (cache_elem_bytes != 1 && cache_elem_bytes != 2)
    return fail(FASTTPS_ERR_INVALID_ARG, "cache_elem_bytes %d: 2 (bf16) or 1 (8-bit codes)", cache_elem_bytes);
  int maxp = 0;
  return check_args(*cfg, x, pos, batch, k_cache, v_cache, y, &maxp, (size_t)cache_elem_bytes);
}

}  // extern "C"

namespace {

// Attention split: the tiles of 64 cached positions [0, pos) of every
// (sequence, kv head) are dealt to nsplit interleaved splits of about
// split_len positions, so that about `target` blocks carry the work (the new
// entry at pos comes from registers, so it adds no tile of its own).
int attention_splits(const fasttps_layer* l, const int32_t* pos, int32_t batch, int maxp) {
  const fasttps_config& c = l->cfg;
  const int maxn = std::max(maxp, 1);
  long total = 0;
  int minp = maxp;
  for (int b = 0; b < batch; ++b) {
    total += pos[b];
    minp = std::min(minp, (int)pos[b]);
  }
  const long target =
      batch == 1 ? kTargetAttnBlocksOne : (minp == maxp ? 1 : kRaggedAttnFactor) * (long)kTargetAttnBlocks;
  int split_len = round_up((int)std::min<long>((total * c.n_kv_heads + target - 1) / target, maxn), kAttnTile);
  split_len = std::max(split_len, round_up(ceil_div(maxn, l->nsplit_cap), kAttnTile));
  return ceil_div(maxn, split_len);
}

// Where a step keeps its fp32 intermediates: the layer handle's scratch, or
// (the allocation-free step) the static array, with the split partials laid
// out for exactly the step's nsplit splits.
struct StepScratch {
  float* qkv;
  float* part;
  float* o;
  float* h1;
  float* a;
  int nsplit_cap;
  bool noalloc;  // the vector path only, no test hooks, no timing events
};

// Bytes of static scratch a step of `batch` sequences with nsplit splits
// needs, and the layout (offsets in floats) if `out` is set.
size_t noalloc_layout(const fasttps_config& c, int batch, int nsplit, float* base, StepScratch* out) {
  const size_t B = batch, d = c.head_dim;
  const size_t sizes[5] = {B * (c.n_heads + 2 * c.n_kv_heads) * d * sizeof(float),
                           B * c.n_heads * nsplit * (d + kPartLead) * sizeof(float), B * c.n_heads * d * sizeof(float),
                           B * c.hidden * sizeof(float), B * c.intermediate * sizeof(float)};
  size_t offs[5], total = 0;
  for (int i = 0; i < 5; ++i) {
    offs[i] = total;
    total += align256(sizes[i]);
  }
  if (out) {
    char* p = reinterpret_cast<char*>(base);
    *out = StepScratch{reinterpret_cast<float*>(p + offs[0]), reinterpret_cast<float*>(p + offs[1]),
                       reinterpret_cast<float*>(p + offs[2]), reinterpret_cast<float*>(p + offs[3]),
                       reinterpret_cast<float*>(p + offs[4]), nsplit, true};
  }
  return total;
}

// The fused step after validation: kvf is the cache format (kKvBf16, or an
// 8-bit format with its scales in *sc); scr overrides the layer's scratch.
int run_step(fasttps_layer* l, const fasttps_weights* w, const void* x, const int32_t* pos, int32_t batch,
             void* k_cache, void* v_cache, void* y, void* stream, int maxp, int kvf, const KvScales* sc,
             const StepScratch* scr = nullptr) {
  const fasttps_config& c = l->cfg;
  const size_t D = c.hidden, d = c.head_dim;
  const StepScratch own{l->qkv, l->attn_part, l->attn_o, l->h1, l->mlp_a, l->nsplit_cap, false};
  const StepScratch& S = scr ? *scr : own;
  // projections on the matrix cores from kMfmaMinBatch sequences up (or as
  // fasttps_set_gemm_path says), where the weights carry MFMA tiles; the
  // allocation-free step runs the vector path
  const bool have_tiles = w->t_qkv != nullptr && l->op_o != nullptr;
  // the fused MLP runs with the vector projections (and not in the
  // allocation-free step)
  const bool mlp_fused = !S.noalloc && l->mlp_path == FASTTPS_MLP_FUSED;
  if (mlp_fused && !w->w_down_slices)
    return fail(FASTTPS_ERR_INVALID_ARG, "the fused MLP needs weights packed while it was selected on the layer");
  // weights in the tile order only run the matrix path, at any batch
  const bool tiles_only = w->w_qkv == nullptr;
  if (tiles_only && (S.noalloc || mlp_fused || l->gemm_path == FASTTPS_GEMM_VECTOR ||
                     l->gemm_path == FASTTPS_GEMM_FUSED))
    return fail(FASTTPS_ERR_INVALID_ARG,
                "weights packed in the tile order only (FASTTPS_WEIGHTS_TILES) run the matrix path only");
  const bool mfma = !S.noalloc && !mlp_fused &&
                    (l->gemm_path == FASTTPS_GEMM_MATRIX || tiles_only ||
                     (l->gemm_path == FASTTPS_GEMM_AUTO && have_tiles && batch >= kMfmaMinBatch));
  if (mfma && !have_tiles)
    return fail(FASTTPS_ERR_INVALID_ARG, "the matrix-core path needs a layer and weights with max_batch > 1");

  const int nsplit = attention_splits(l, pos, batch, maxp);

  // one sequence: the whole step as one persistent kernel, on request
  // (FASTTPS_GEMM_FUSED), where it is built for the shape and the step is the
  // plain bf16-cache step. Not the automatic choice: on MI355X its phase
  // hand-overs through coherent flags cost more than the separate kernels'
  // boundaries in a HIP graph (69.6 vs 54.4 us per Phi-3 layer at KV 4096).
  FusedShape fsh{};
  fsh.head_dim = (int)d;
  fsh.group = c.n_heads / c.n_kv_heads;
  fsh.q = gemv_shape_b1((int)D, false);
  fsh.o = gemv_shape_b1(c.n_heads * (int)d, false);
  fsh.gu = gemv_shape_b1((int)D, true);
  fsh.down = gemv_shape_b1(c.intermediate, false);
  const bool fused_ok = batch == 1 && kvf == kKvBf16 && l->p_bf16 == 0 && nsplit <= fused_layer_max_splits() &&
                        nsplit * c.n_kv_heads <= fused_layer_grid() && c.n_heads * (int)d <= 4096 &&
                        fused_layer_supported(fsh);
  const bool fused = !mfma && !S.noalloc && !mlp_fused && l->gemm_path == FASTTPS_GEMM_FUSED;
  if (fused && !fused_ok)
    return fail(FASTTPS_ERR_UNSUPPORTED, "the fused kernel is built for one sequence of the Phi-3-mini layer shape");

  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != l->device) return fail(FASTTPS_ERR_INVALID_ARG, "current device %d is not the layer's device %d", dev, l->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint16_t* xb = static_cast<const uint16_t*>(x);
  KernelEvents ev[FASTTPS_NUM_KERNELS];
  const bool timed = !S.noalloc && l->prof_n < l->prof_cap;
  const bool debug = !S.noalloc && l->debug;
  if (timed) {
    for (int k = 0; k < FASTTPS_NUM_KERNELS; ++k) {
      const size_t i = ((size_t)l->prof_n * FASTTPS_NUM_KERNELS + k) * 2;
      ev[k].start = l->prof_events[i];
      ev[k].stop = l->prof_events[i + 1];
    }
  }
  auto used = [&](int k) {
    if (timed) l->prof_used[(size_t)l->prof_n * FASTTPS_NUM_KERNELS + k] = 1;
  };

  // the vector path's arguments (also the fused kernel's phases)
  GemvArgs qa{};
  qa.w = w->w_qkv;
  qa.rows = (c.n_heads + 2 * c.n_kv_heads) * (int)d;
  qa.din = (int)D;
  qa.batch = batch;
  qa.x_bf16 = xb;
  qa.gamma = w->attn_norm;
  qa.out = S.qkv;
  qa.eps = c.rms_eps;
  qa.dbg_act = debug ? l->dbg_h : nullptr;
  GemvArgs oa{};
  oa.w = w->w_o;
  oa.rows = (int)D;
  oa.din = c.n_heads * (int)d;
  oa.batch = batch;
  oa.x_bf16 = xb;
  oa.in_f32 = S.o;
  oa.out = S.h1;
  oa.eps = c.rms_eps;
  GemvArgs ga{};
  ga.w = w->w_gu;
  ga.rows = c.intermediate;
  ga.din = (int)D;
  ga.batch = batch;
  ga.gamma = w->mlp_norm;
  ga.in_f32 = S.h1;
  ga.out = S.a;
  ga.eps = c.rms_eps;
  ga.dbg_act = debug ? l->dbg_h2 : nullptr;
  GemvArgs da{};
  da.w = w->w_down;
  da.rows = (int)D;
  da.din = c.intermediate;
  da.batch = batch;
  da.in_f32 = S.a;
  da.res_f32 = S.h1;
  da.out_bf16 = static_cast<uint16_t*>(y);
  da.eps = c.rms_eps;

  AttnArgs aa{};
  aa.qkv = S.qkv;
  aa.rope_cos = l->rope_cos;
  aa.rope_sin = l->rope_sin;
  aa.k_cache = static_cast<uint16_t*>(k_cache);
  aa.v_cache = static_cast<uint16_t*>(v_cache);
  aa.part = S.part;
  aa.o = S.o;
  aa.o_operand = mfma ? l->op_o : nullptr;
  aa.o_nbtc = l->nbtc;
  aa.batch = batch;
  aa.n_heads = c.n_heads;
  aa.n_kv_heads = c.n_kv_heads;
  aa.head_dim = (int)d;
  aa.max_seq = c.max_seq;
  aa.nsplit = nsplit;
  aa.nsplit_cap = S.nsplit_cap;
  aa.scale = (float)(1.0 / std::sqrt((double)d));
  aa.p_bf16 = l->p_bf16;
  aa.kv_format = kvf;
  aa.dbg_qk = debug ? l->dbg_qk : nullptr;
  for (int b = 0; b < batch; ++b) aa.pos.p[b] = pos[b];
  // the longest sequences' blocks first (ties in batch order)
  for (int b = 0; b < batch; ++b) aa.order.p[b] = b;
  std::stable_sort(aa.order.p, aa.order.p + batch, [&](int32_t u, int32_t v) { return pos[u] > pos[v]; });

  if (!S.noalloc) {
    l->dbg_written = 0;
    l->mlp_a_written = !mlp_fused;  // h^sm is stored by every path but the fused MLP
  }
  if (fused) {
    FusedArgs f{};
    f.qkv = qa;
    f.oproj = oa;
    f.gateup = ga;
    f.down = da;
    f.attn = aa;
    // the one-kernel step has no test-hook outputs
    f.qkv.dbg_act = f.gateup.dbg_act = nullptr;
    f.attn.dbg_qk = nullptr;
    f.flags = l->fused_flags;
    f.epoch = l->fused_epoch;
    f.err = l->fused_err;
    f.attn_items = nsplit * c.n_kv_heads;
    f.stage_floats = std::max({c.n_heads * (int)d, (int)D, c.intermediate});
    if ((e = launch_fused_layer(f, fsh, s, ev[6])) != hipSuccess) return hip_fail(e, "fused layer launch");
    used(6);
    if (timed) ++l->prof_n;
    return FASTTPS_OK;
  }

  const LayerTiles lt = layer_tiles(c);
  auto mfma_args = [&](const TileDims& td, const uint16_t* wt, int rows, int din) {
    MfmaArgs m{};
    m.w = wt;
    m.ns = td.ns;
    m.kt = td.kt;
    m.rh = td.rh;
    m.nt = ceil_div(td.kt, kMfmaWaves);
    m.rows = rows;
    m.din = din;
    m.batch = batch;
    m.nbtc = l->nbtc;
    m.a_out_nbtc = l->nbtc;
    m.eps = c.rms_eps;
    m.kpart = l->split_part;
    m.tickets = l->split_tickets;
    m.kpart_cap = l->split_part_cap;
    m.tickets_cap = l->split_tickets_cap;
    return m;
  };

  if (mfma) {
    MfmaArgs m = mfma_args(lt.qkv, w->t_qkv, qa.rows, (int)D);
    m.x_bf16 = xb;
    m.gamma = w->attn_norm;
    m.out = S.qkv;
    if ((e = launch_mfma_qkv(m, s, ev[0])) != hipSuccess) return hip_fail(e, "qkv launch");
  } else {
    if ((e = launch_rmsnorm_qkv(qa, s, ev[0])) != hipSuccess) return hip_fail(e, "qkv launch");
  }
  used(0);

  e = kvf == kKvBf16 ? launch_attention(aa, s, ev[1]) : launch_attention_kv8(aa, *sc, s, ev[1]);
  if (e != hipSuccess) return hip_fail(e, "attention launch");
  used(1);
  // one sequence on the vector path: the O projection merges the splits in
  // its prologue, one launch fewer (Phi-3 layer on MI355X, HIP graph: 60.1 ->
  // 57.8 us per step at KV 4096, 54.5 -> 52.0 us at KV 1024); otherwise the
  // combine kernel
  const bool merge_in_o = !mfma && batch == 1 && oproj_merge_supported(c.n_heads, (int)d, nsplit, (int)D);
  if (!merge_in_o) {
    if ((e = launch_attention_combine(aa, s, ev[2])) != hipSuccess) return hip_fail(e, "attention combine launch");
    used(2);
  }

  if (mfma) {
    MfmaArgs m = mfma_args(lt.o, w->t_o, (int)D, c.n_heads * (int)d);
    m.x_bf16 = xb;
    m.gamma = w->mlp_norm;
    m.a_in = l->op_o;
    m.out = S.h1;
    m.a_out = l->op_gu;
    m.ssq_out = l->ssq_h1;
    if ((e = launch_mfma_oproj(m, s, ev[3])) != hipSuccess) return hip_fail(e, "o-proj launch");
    m = mfma_args(lt.gu, w->t_gu, c.intermediate, (int)D);
    m.a_in = l->op_gu;
    m.ssq_in = l->ssq_h1;
    m.ns_in = lt.o.ns;
    m.out = S.a;
    m.a_out = l->op_down;
    if ((e = launch_mfma_gate_up(m, s, ev[4])) != hipSuccess) return hip_fail(e, "mlp gate/up launch");
    m = mfma_args(lt.down, w->t_down, (int)D, c.intermediate);
    m.a_in = l->op_down;
    m.res_f32 = S.h1;
    m.out_bf16 = static_cast<uint16_t*>(y);
    if ((e = launch_mfma_down(m, s, ev[5])) != hipSuccess) return hip_fail(e, "mlp down launch");
  } else {
    if (merge_in_o) {
      MergeArgs ma{};
      ma.part = S.part;
      ma.o = S.o;
      ma.nsplit = nsplit;
      ma.nsplit_cap = S.nsplit_cap;
      ma.n_heads = c.n_heads;
      ma.head_dim = (int)d;
      if ((e = launch_oproj_merge(oa, ma, s, ev[3])) != hipSuccess) return hip_fail(e, "o-proj launch");
    } else if ((e = launch_oproj_residual(oa, s, ev[3])) != hipSuccess) {
      return hip_fail(e, "o-proj launch");
    }
    if (mlp_fused) {
      MlpFusedArgs mf{};
      mf.w_down_slices = w->w_down_slices;
      mf.part = l->mlp_part;
      mf.y = static_cast<uint16_t*>(y);
      mf.nblk = mlp_fused_blocks(c.intermediate);
      mf.u8 = mlp_fused_u8(c.intermediate);
      mf.hidden = (int)D;
      mf.batch = batch;
      if ((e = launch_mlp_fused(ga, mf, s, ev[4], ev[5])) != hipSuccess) return hip_fail(e, "fused mlp launch");
    } else {
      if ((e = launch_gate_up(ga, s, ev[4])) != hipSuccess) return hip_fail(e, "mlp gate/up launch");
      if ((e = launch_down_residual(da, s, ev[5])) != hipSuccess) return hip_fail(e, "mlp down launch");
    }
  }
  used(3);
  used(4);
  used(5);
  if (timed) ++l->prof_n;
  if (debug) l->dbg_written = kDbgQk | (mfma ? 0 : kDbgNorm);
  return FASTTPS_OK;
}

}  // namespace

extern "C" {

int fasttps_decode_step(fasttps_layer* l, const fasttps_weights* w, const void* x, const int32_t* pos,
                        int32_t batch, void* k_cache, void* v_cache, void* y, void* stream) {
  g_last_error.clear();
  int maxp = 0;
  const int st = check_step(l, w, x, pos, batch, k_cache, v_cache, y, &maxp);
  if (st) return st;
  return run_step(l, w, x, pos, batch, k_cache, v_cache, y, stream, maxp, kKvBf16, nullptr);
}

int fasttps_decode_step_noalloc(fasttps_layer* l, const fasttps_weights* w, const void* x, const int32_t* pos,
                                int32_t batch, void* k_cache, void* v_cache, void* y, void* stream) {
  g_last_error.clear();
  int maxp = 0;
  const int st = check_step(l, w, x, pos, batch, k_cache, v_cache, y, &maxp);
  if (st) return st;
  const int nsplit = attention_splits(l, pos, batch, maxp);
  const size_t need = noalloc_layout(l->cfg, batch, nsplit, nullptr, nullptr);
  if (need > kStaticScratchBytes)
    return fail(FASTTPS_ERR_UNSUPPORTED,
                "the allocation-free step needs %zu bytes of scratch for %d sequences; its static buffer holds %zu",
                need, batch, kStaticScratchBytes);
  float* base = static_cast<float*>(static_scratch(l->device));
  if (!base) return fail(FASTTPS_ERR_HIP, "no static scratch address for device %d", l->device);
  StepScratch scr{};
  noalloc_layout(l->cfg, batch, nsplit, base, &scr);
  return run_step(l, w, x, pos, batch, k_cache, v_cache, y, stream, maxp, kKvBf16, nullptr, &scr);
}

int fasttps_decode_step_kv8(fasttps_layer* l, const fasttps_weights* w, const void* x, const int32_t* pos,
                            int32_t batch, int32_t kv_format, void* k_cache, void* v_cache, const float* k_scale,
                            const float* v_scale, void* y, void* stream) {
  g_last_error.clear();
  if (kv_format != FASTTPS_KV_FP8_E4M3 && kv_format != FASTTPS_KV_INT8)
    return fail(FASTTPS_ERR_INVALID_ARG, "unknown KV format %d", kv_format);
  int maxp = 0;
  const int st = check_step(l, w, x, pos, batch, k_cache, v_cache, y, &maxp, 1);
  if (st) return st;
  if (!k_scale || !v_scale) return fail(FASTTPS_ERR_INVALID_ARG, "null scale array");
  const int Hkv = l->cfg.n_kv_heads;
  if (Hkv > kMaxKvHeads) return fail(FASTTPS_ERR_UNSUPPORTED, "n_kv_heads %d > %d", Hkv, kMaxKvHeads);
  KvScales sc{};
  for (int g = 0; g < Hkv; ++g) {
    if (!(std::isfinite(k_scale[g]) && k_scale[g] > 0.f) || !(std::isfinite(v_scale[g]) && v_scale[g] > 0.f))
      return fail(FASTTPS_ERR_INVALID_ARG, "KV head %d: scales must be positive and finite", g);
    sc.k[g] = k_scale[g];
    sc.v[g] = v_scale[g];
  }
  static_assert(FASTTPS_KV_FP8_E4M3 == kKvFp8 && FASTTPS_KV_INT8 == kKvInt8, "format codes");
  const int kvf = kv_format;
  return run_step(l, w, x, pos, batch, k_cache, v_cache, y, stream, maxp, kvf, &sc);
}

int fasttps_debug_read(fasttps_layer* l, int32_t which, int32_t batch, void* dst, size_t bytes, void* stream) {
  g_last_error.clear();
  if (!layer_ok(l)) return fail(FASTTPS_ERR_BAD_HANDLE, "bad layer handle");
  if (!dst) return fail(FASTTPS_ERR_INVALID_ARG, "dst is null");
  const fasttps_config& c = l->cfg;
  if (batch < 1 || batch > c.max_batch) return fail(FASTTPS_ERR_INVALID_ARG, "batch out of range");
  const void* src = nullptr;
  size_t n = 0;
  switch (which) {
    case FASTTPS_DBG_QKV: src = l->qkv; n = (size_t)(c.n_heads + 2 * c.n_kv_heads) * c.head_dim; break;
    case FASTTPS_DBG_ATTN: src = l->attn_o; n = (size_t)c.n_heads * c.head_dim; break;
    case FASTTPS_DBG_H1: src = l->h1; n = (size_t)c.hidden; break;
    case FASTTPS_DBG_MLP_A:
      if (!l->mlp_a_written)
        return fail(FASTTPS_ERR_INVALID_ARG, "the last step kept h^sm on chip (fused MLP): nothing to read");
      src = l->mlp_a;
      n = (size_t)c.intermediate;
      break;
    case FASTTPS_DBG_FUSED_WAITS: src = l->fused_err; n = 1; batch = 1; break;
    case FASTTPS_DBG_QK_ROPE:
    case FASTTPS_DBG_H:
    case FASTTPS_DBG_H2: {
      const int need = which == FASTTPS_DBG_QK_ROPE ? kDbgQk : kDbgNorm;
      if (!(l->dbg_written & need))
        return fail(FASTTPS_ERR_INVALID_ARG,
                    "debug buffer %d was not written by the last step (fasttps_set_debug off, the one-kernel "
                    "step, or for the normalized activations a matrix-core step)", which);
      src = which == FASTTPS_DBG_QK_ROPE ? l->dbg_qk : which == FASTTPS_DBG_H ? l->dbg_h : l->dbg_h2;
      n = which == FASTTPS_DBG_QK_ROPE ? (size_t)(c.n_heads + c.n_kv_heads) * c.head_dim : (size_t)c.hidden;
      break;
    }
    default: return fail(FASTTPS_ERR_INVALID_ARG, "unknown debug buffer %d", which);
  }
  n *= (size_t)batch * sizeof(float);
  if (bytes != n) return fail(FASTTPS_ERR_INVALID_ARG, "bytes %zu != %zu", bytes, n);
  hipError_t e = hipMemcpyAsync(dst, src, n, hipMemcpyDeviceToDevice, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "debug copy");
  return FASTTPS_OK;
}

}  // extern "C"

int fasttps_unfused_enable(fasttps_layer* l) {
  g_last_error.clear();
  if (!layer_ok(l)) return fail(FASTTPS_ERR_BAD_HANDLE, "bad layer handle");
  if (l->uf_arena) return FASTTPS_OK;
  const fasttps_config& c = l->cfg;
  const size_t B = c.max_batch, D = c.hidden, H = c.n_heads, Hkv = c.n_kv_heads, d = c.head_dim;
  const size_t K = c.intermediate, N = c.max_seq;
  const int pv_cap = unfused_pv_splits(c.max_seq);
  // fp32 buffers, then the two bf16 concat buffers
  const size_t f32[] = {B * D,       B * H * d, B * Hkv * d, B * Hkv * d, B * H * d, B * Hkv * d, B * H * d,
                        B * Hkv * d, B * Hkv * d, B * H * N,  B * H * N,   B * H * (size_t)pv_cap * d,
                        B * H * d,   B * D,     B * D,       B * D,       B * K,     B * K,       B * K,
                        B * K,       B * D};
  constexpr int kF = sizeof(f32) / sizeof(f32[0]);
  size_t offs[kF + 2], total = 0;
  for (int i = 0; i < kF; ++i) {
    offs[i] = total;
    total += align256(f32[i] * sizeof(float));
  }
  const size_t cat_bytes = B * Hkv * N * d * sizeof(uint16_t);
  offs[kF] = total;
  total += align256(cat_bytes);
  offs[kF + 1] = total;
  total += align256(cat_bytes);
  void* arena = nullptr;
  hipError_t e = hipMalloc(&arena, total);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(FASTTPS_ERR_OOM, "hipMalloc(%zu): %s", total, hipGetErrorString(e));
  }
  char* base = static_cast<char*>(arena);
  float* p[kF];
  for (int i = 0; i < kF; ++i) p[i] = reinterpret_cast<float*>(base + offs[i]);
  UnfusedArgs& u = l->uf;
  u.h = p[0]; u.q = p[1]; u.k = p[2]; u.v = p[3]; u.q_rope = p[4]; u.k_rope = p[5]; u.q_t = p[6];
  u.k_t = p[7]; u.v_t = p[8]; u.S = p[9]; u.P = p[10]; u.pv_part = p[11]; u.O = p[12]; u.attn_out = p[13];
  u.h1 = p[14]; u.h2 = p[15]; u.g = p[16]; u.sg = p[17]; u.up = p[18]; u.hp = p[19]; u.mlp_out = p[20];
  u.kcat = reinterpret_cast<uint16_t*>(base + offs[kF]);
  u.vcat = reinterpret_cast<uint16_t*>(base + offs[kF + 1]);
  u.pv_cap = pv_cap;
  l->uf_arena = arena;
  return FASTTPS_OK;
}

int fasttps_decode_step_unfused(fasttps_layer* l, const fasttps_weights* w, const void* x, const int32_t* pos,
                                int32_t batch, void* k_cache, void* v_cache, void* y, void* stream) {
  g_last_error.clear();
  int maxp = 0;
  const int st = check_step(l, w, x, pos, batch, k_cache, v_cache, y, &maxp);
  if (st) return st;
  if (!l->uf_arena) return fail(FASTTPS_ERR_INVALID_ARG, "call fasttps_unfused_enable on this layer first");
  if (!w->w_qkv)
    return fail(FASTTPS_ERR_INVALID_ARG, "the op-by-op baseline needs row-major weights (FASTTPS_WEIGHTS_TILES set)");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != l->device) return fail(FASTTPS_ERR_INVALID_ARG, "current device %d is not the layer's device %d", dev, l->device);
  const fasttps_config& c = l->cfg;
  UnfusedArgs u = l->uf;
  u.x = static_cast<const uint16_t*>(x);
  u.attn_norm = w->attn_norm;
  u.mlp_norm = w->mlp_norm;
  u.w_qkv = w->w_qkv;
  u.w_o = w->w_o;
  u.w_gu = w->w_gu;
  u.w_down = w->w_down;
  u.k_cache = static_cast<uint16_t*>(k_cache);
  u.v_cache = static_cast<uint16_t*>(v_cache);
  u.y = static_cast<uint16_t*>(y);
  u.rope_cos = l->rope_cos;
  u.rope_sin = l->rope_sin;
  u.batch = batch;
  u.hidden = c.hidden;
  u.n_heads = c.n_heads;
  u.n_kv_heads = c.n_kv_heads;
  u.head_dim = c.head_dim;
  u.inter = c.intermediate;
  u.max_seq = c.max_seq;
  u.maxn = maxp + 1;
  u.scale = (float)(1.0 / std::sqrt((double)c.head_dim));
  u.eps = c.rms_eps;
  for (int b = 0; b < batch; ++b) u.pos.p[b] = pos[b];
  if ((e = launch_unfused(u, static_cast<hipStream_t>(stream))) != hipSuccess) return hip_fail(e, "unfused launch");
  return FASTTPS_OK;
}

int fasttps_set_weight_layout(fasttps_layer* l, int32_t layout) {
  g_last_error.clear();
  if (!layer_ok(l)) return fail(FASTTPS_ERR_BAD_HANDLE, "bad layer handle");
  if (layout != FASTTPS_WEIGHTS_ROWS_AND_TILES && layout != FASTTPS_WEIGHTS_TILES)
    return fail(FASTTPS_ERR_INVALID_ARG, "unknown weight layout %d", layout);
  if (layout == FASTTPS_WEIGHTS_TILES && !l->op_o)
    return fail(FASTTPS_ERR_INVALID_ARG, "the tile order only needs a layer with max_batch > 1");
  l->weight_layout = layout;
  return FASTTPS_OK;
}

int fasttps_set_gemm_path(fasttps_layer* l, int32_t path) {
  g_last_error.clear();
  if (!layer_ok(l)) return fail(FASTTPS_ERR_BAD_HANDLE, "bad layer handle");
  if (path != FASTTPS_GEMM_AUTO && path != FASTTPS_GEMM_VECTOR && path != FASTTPS_GEMM_MATRIX &&
      path != FASTTPS_GEMM_FUSED)
    return fail(FASTTPS_ERR_INVALID_ARG, "unknown projection path %d", path);
  if (path == FASTTPS_GEMM_MATRIX && !l->op_o)
    return fail(FASTTPS_ERR_INVALID_ARG, "the matrix-core path needs a layer with max_batch > 1");
  l->gemm_path = path;
  return FASTTPS_OK;
}

int fasttps_set_mlp_path(fasttps_layer* l, int32_t path) {
  g_last_error.clear();
  if (!layer_ok(l)) return fail(FASTTPS_ERR_BAD_HANDLE, "bad layer handle");
  if (path != FASTTPS_MLP_SPLIT && path != FASTTPS_MLP_FUSED)
    return fail(FASTTPS_ERR_INVALID_ARG, "unknown MLP path %d", path);
  if (path == FASTTPS_MLP_FUSED && !l->mlp_part) {
    const fasttps_config& c = l->cfg;
    const size_t bytes = (size_t)mlp_fused_blocks(c.intermediate) * c.max_batch * c.hidden * sizeof(float);
    void* p = nullptr;
    const hipError_t e = hipMalloc(&p, bytes);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(FASTTPS_ERR_OOM, "hipMalloc(%zu): %s", bytes, hipGetErrorString(e));
    }
    l->mlp_part = static_cast<float*>(p);
  }
  l->mlp_path = path;
  return FASTTPS_OK;
}

int fasttps_set_debug(fasttps_layer* l, int32_t enable) {
  g_last_error.clear();
  if (!layer_ok(l)) return fail(FASTTPS_ERR_BAD_HANDLE, "bad layer handle");
  l->debug = enable ? 1 : 0;
  return FASTTPS_OK;
}

int fasttps_set_attention_p_bf16(fasttps_layer* l, int32_t enable) {
  g_last_error.clear();
  if (!layer_ok(l)) return fail(FASTTPS_ERR_BAD_HANDLE, "bad layer handle");
  l->p_bf16 = enable ? 1 : 0;
  return FASTTPS_OK;
}
