// Host runtime of the sparse-depth verification step: the C ABI of tss.h.
//
// It owns no device memory.  It validates inputs, packs weights into the
// caller's buffer, keeps per-sequence KV bookkeeping (committed length and,
// per layer, how many committed rows hold K/V), derives tree metadata, and
// enqueues the kernels on the caller's stream.  The skip rule of the paper's
// Domain-Aware Skip Controller (before block l, check l against the skip set;
// a skipped block passes the hidden state through) is applied here: the layer
// loop launches nothing for a skipped block, so its weights and KV pages are
// never read or written.
#include "../../include/tss.h"
#include "tss_internal.h"

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <string>
#include <thread>
#include <vector>

using namespace tss;

namespace tss {
LaunchTiming& launch_timing() {
  static thread_local LaunchTiming t;
  return t;
}
}  // namespace tss

namespace {

constexpr size_t kStageBytes = 32u << 20;  // one pinned weight-upload buffer

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct LayerW {
  size_t attn_norm, qkv, o, mlp_norm, gateup, down;
};

struct WeightLayout {
  size_t embed = 0, final_norm = 0, lm_head = 0, total = 0;
  std::vector<LayerW> layers;
};

struct WsLayout {
  size_t sp, result, h, xa, xm, ss_a, ss_m, q, o, act, part_o, part_ml, counters, attn_split, kpart, kcount, acount, logits,
      am_val, am_idx, greedy, total;
  int n_counters;
};

// weight element bytes; the KV cache uses the same width (fp16 in the bf16
// mode, fp32 in the f32 mode)
int elem_size(const tss_model_cfg* c) { return c->dtype == TSS_BF16 ? 2 : 4; }
// activation planes: one fp16 plane in the bf16-weight mode, one fp32 plane
// otherwise
int act_planes(const tss_model_cfg*) { return 1; }

// A bf16 bit pattern as the fp16 bit pattern of the same value, rounded to
// nearest even.  bf16 keeps 7 fraction bits and fp16 10, so every normal fp16
// value is exact: exponents 2^-14 .. 2^15 map across unchanged.  Below 2^-14
// the value (1.m * 2^(e-127), as an integer (128 + m) in units of 2^(e-134))
// becomes a multiple of fp16's subnormal unit 2^-24 with a rounded right
// shift.  Finite values from 65536 up (no fp16 value of the same magnitude)
// set *over and become infinity; infinities and NaNs (kept quiet) map across.
uint16_t bf16_bits_to_f16(uint16_t b, bool* over) {
  const uint16_t sign = b & 0x8000u;
  const uint32_t e = (b >> 7) & 0xffu, m = b & 0x7fu;
  if (e == 0xff) return sign | 0x7c00u | (m ? 0x200u | (m << 3) : 0u);
  if (e >= 143) {
    *over = true;
    return sign | 0x7c00u;
  }
  if (e >= 113) return sign | (uint16_t)(((e - 112) << 10) | (m << 3));
  if (e == 0) return sign;  // bf16 subnormals lie below 2^-126
  const uint32_t v = 128u + m;  // value = v * 2^(e - 134), unit 2^-24 for e = 110
  if (e >= 110) return sign | (uint16_t)(v << (e - 110));
  const uint32_t k = 110 - e;
  if (k > 9) return sign;  // below half of 2^-24
  uint32_t q = v >> k;
  const uint32_t r = v & ((1u << k) - 1), half = 1u << (k - 1);
  q += (r > half || (r == half && (q & 1u))) ? 1u : 0u;
  return sign | (uint16_t)q;
}

// The whole map as a table (128 KiB, built once): weight uploads convert
// through it at about one load per element.
const uint16_t* f16_table() {
  static const std::vector<uint16_t> tab = [] {
    std::vector<uint16_t> t(65536);
    bool over = false;
    for (uint32_t b = 0; b < 65536; ++b) t[b] = bf16_bits_to_f16((uint16_t)b, &over);
    return t;
  }();
  return tab.data();
}

// Finite with magnitude >= 65536 (bf16 0x4780): no fp16 value is that large.
bool bf16_out_of_f16_range(uint16_t b) {
  const uint16_t a = b & 0x7fffu;
  return a >= 0x4780u && a < 0x7f80u;
}

// Copies n_bytes of 16-bit weights, converting bf16 to fp16 when to_f16 is
// set; clears *ok on a finite value beyond fp16's range.
void copy_weights(uint8_t* dst, const uint8_t* src, size_t n_bytes, bool to_f16, std::atomic<bool>* ok) {
  if (!to_f16) {
    std::memcpy(dst, src, n_bytes);
    return;
  }
  const uint16_t* tab = f16_table();
  bool over = false;
  for (size_t i = 0; i < n_bytes; i += 2) {
    uint16_t b;
    std::memcpy(&b, src + i, 2);
    over |= bf16_out_of_f16_range(b);
    const uint16_t h = tab[b];
    std::memcpy(dst + i, &h, 2);
  }
  if (over) ok->store(false);
}
int round16(int x) { return (x + 15) & ~15; }
// rows one step can carry: the nodes of every sequence of a batch (the GEMMs
// take up to 8 sixteen-row tiles in the bf16 mode, 4 in the f32 mode)
int row_cap(const tss_model_cfg* c) {
  return std::min(c->max_nodes * c->max_batch, c->dtype == TSS_BF16 ? kMaxRows : 64);
}
// Attention workgroups per (head, item) when a launch has n_items items: at
// most about kAttnTargetWGs workgroups in all (at least one per pair).
int attn_groups(int n_heads, int n_items) {
  return std::max(1, std::min(kAttnMaxGroups, kAttnTargetWGs / (n_heads * n_items)));
}
// Workgroups per (head, item) of a launch whose items come from n_items
// different KV sequences (pages_per_seq pages each at most): one per
// kAttnPagesPerWG pages of the longest possible context, within
// kAttnBatchSlots partial-state slots.
int attn_batch_groups(int n_heads, int n_items, int pages_per_seq) {
  const int by_pages = (pages_per_seq + kAttnPagesPerWG - 1) / kAttnPagesPerWG;
  return std::max(1, std::min(kAttnMaxGroups, std::min(by_pages, kAttnBatchSlots / (n_heads * n_items))));
}
// partial-state slots of one attention launch: n_heads * n_items * groups
// over every item count (at most max(kAttnTargetWGs, n_heads * n_items)),
// and up to kAttnBatchSlots when the context serves batches of sequences
size_t attn_slots(const tss_model_cfg* c) {
  size_t m = 0;
  for (int n = 1; n <= kAttnMaxItems; ++n) m = std::max(m, (size_t)c->n_heads * n * attn_groups(c->n_heads, n));
  if (c->max_batch > 1) m = std::max(m, (size_t)kAttnBatchSlots);
  return m;
}

int cfg_ok(const tss_model_cfg* c) {
  if (!c) return 0;
  if (c->n_layers < 1 || c->n_layers > kMaxLayers) return 0;
  if (c->head_dim != 64 && c->head_dim != 128) return 0;
  if (c->n_heads < 1 || c->d_model != c->n_heads * c->head_dim) return 0;
  if (c->d_model % 32 || c->ffn_dim < 32 || c->ffn_dim % 32 || c->vocab < 32 || c->vocab % 32) return 0;
  if (c->d_model > 8192) return 0;  // RMSNorm partial sums: at most 512 per row
  if (c->dtype != TSS_F32 && c->dtype != TSS_BF16) return 0;
  if (c->max_nodes < 1 || c->max_nodes > kMaxNodes) return 0;
  if (c->max_batch < 1 || c->max_batch > kMaxBatch) return 0;
  if (c->dtype == TSS_F32 && c->d_model > 4096) return 0;  // the fp32 mode serves small models; validated up to 4096
  if (!(c->rms_eps > 0.f) || !(c->rope_base > 1.f)) return 0;
  return 1;
}

WeightLayout weight_layout(const tss_model_cfg* c) {
  WeightLayout w;
  const size_t es = elem_size(c), d = c->d_model, f = c->ffn_dim, v = c->vocab;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align256(off + bytes); return o; };
  w.embed = take(v * d * es);
  w.layers.resize(c->n_layers);
  for (auto& L : w.layers) {
    L.attn_norm = take(d * 4);
    L.qkv = take(3 * d * d * es);
    L.o = take(d * d * es);
    L.mlp_norm = take(d * 4);
    L.gateup = take(2 * f * d * es);
    L.down = take(d * f * es);
  }
  w.final_norm = take(d * 4);
  w.lm_head = take(v * d * es);
  w.total = off;
  return w;
}

WsLayout ws_layout(const tss_model_cfg* c) {
  WsLayout w;
  const size_t es = elem_size(c), d = c->d_model, f = c->ffn_dim, v = c->vocab;
  const size_t Mp = round16(row_cap(c));
  const size_t ap = act_planes(c);
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align256(off + bytes); return o; };
  w.sp = take(sizeof(StepParams));
  w.result = take(kMaxSegs * sizeof(Result));
  w.h = take(Mp * d * 4);
  w.xa = take(ap * Mp * d * es);
  w.xm = take(ap * Mp * d * es);
  w.ss_a = take((d / 16) * Mp * 4);
  w.ss_m = take((d / 16) * Mp * 4);
  w.q = take(Mp * d * 4);
  w.o = take(ap * Mp * d * es);
  w.act = take(ap * Mp * f * es);
  const size_t slots = attn_slots(c);
  w.part_o = take(slots * kAttnMaxTiles * 16 * c->head_dim * 4);
  w.part_ml = take(slots * kAttnMaxTiles * 16 * 2 * 4);
  // arrival counters of the attention merges, of the K-split strips and of
  // the argmax rows, one region that every step clears first (embedding kernel)
  w.counters = take((size_t)c->n_heads * kAttnMaxItems * 4 + (d / 16) * 4 + 4);
  w.kcount = w.counters + (size_t)c->n_heads * kAttnMaxItems * 4;
  w.acount = w.kcount + (d / 16) * 4;
  w.n_counters = c->n_heads * kAttnMaxItems + (int)(d / 16) + 1;
  w.attn_split = take((2 * kAttnMaxItems + 1) * 4);
  w.kpart = take((size_t)kMaxKSplit * d * Mp * 4);  // K-split partial products of the residual projections
  w.logits = take(Mp * v * 4);
  w.am_val = take((v / 16) * Mp * 4);
  w.am_idx = take((v / 16) * Mp * 4);
  w.greedy = take(Mp * 4);
  w.total = off;
  return w;
}

struct KvLayout {
  int pages_per_seq = 0, n_pages = 0;
  size_t page_table = 0, rope = 0, pages = 0, total = 0;
};

KvLayout kv_layout(const tss_model_cfg* c, int n_seqs, int max_tokens) {
  KvLayout k;
  k.pages_per_seq = (max_tokens + kPage - 1) / kPage;
  k.n_pages = n_seqs * k.pages_per_seq;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = align256(off + bytes); return o; };
  k.page_table = take((size_t)k.n_pages * 4);
  k.rope = take((size_t)max_tokens * (c->head_dim / 2) * sizeof(float2));
  k.pages = take((size_t)c->n_layers * k.n_pages * 2 * c->n_heads * kPage * c->head_dim * elem_size(c));
  k.total = off;
  return k;
}

}  // namespace

struct tss_ctx {
  tss_model_cfg cfg{};
  bool bf16 = false;
  int es = 4, Mp = 16, KC = 16;
  hipStream_t stream = nullptr;
  int device = 0;                 // device current at creation (the stream's)
  uint8_t* w = nullptr;
  uint8_t* ws = nullptr;          // workspace of the next step (the caller's, or the static scratch)
  WeightLayout wl;
  WsLayout wsl{};
  int Mp_own = 16;
  uint8_t* ws_own = nullptr;      // the caller's workspace and its layout
  WsLayout wsl_own{};
  const uint8_t* out_ws = nullptr;  // workspace and layout of the last step (logits, greedy, split report)
  WsLayout out_wsl{};
  bool direct_only = false;       // set while a step must not be captured (static scratch)
  // KV pool
  uint8_t* kv = nullptr;
  KvLayout kvl;
  int n_seqs = 0, max_tokens = 0;
  std::vector<int32_t> n_kv;
  std::vector<int32_t> pt_host;   // host copy of the page tables
  std::vector<std::vector<int32_t>> kv_len;
  std::vector<std::vector<uint8_t>> mask;
  // pinned host staging: step parameters and result, and two weight-upload
  // buffers (packing one while the other is copied)
  uint8_t* stage[2] = {nullptr, nullptr};
  hipEvent_t stage_ev[2] = {nullptr, nullptr};
  int stage_cur = 0;
  StepParams* sp_host = nullptr;
  // the step being enqueued: its segments' KV sequences, their masks
  // (n_seqs x n_layers) and which of them need their accepted tree path
  // moved after the commit
  struct Step {
    int n_seqs = 0;  // segments
    int32_t seq[kMaxSegs] = {};
    bool compact[kMaxSegs] = {};
    std::vector<uint8_t> mask;
  } step;
  Result* res_host = nullptr;     // [kMaxSegs] host-mapped, written by the accept kernel
  Result* res_dev_map = nullptr;  // its device address
  int last_M = 0;
  int last_results = 0;  // results (segments) of the last verify step in res_host
  bool poisoned = false;
  std::string err;
  // verify steps replayed from captured HIP graphs, keyed by the step's shape
  struct GraphEntry {
    std::string key;
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    hipGraphNode_t embed_node = nullptr;
    hipKernelNodeParams embed_params{};
    uint64_t last_use = 0;
  };
  int launch_mode = TSS_LAUNCH_GRAPH;
  hipStream_t cap_stream = nullptr;
  std::vector<GraphEntry> graphs;
  uint64_t graph_clock = 0;
  hipStream_t cur_stream = nullptr;  // stream the launches of the current step go to
  // one-launch event timing
  int prof_kind = -1, prof_layer = -1;
  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  bool prof_armed = false;
  double prof_ms = 0.0;
  int64_t prof_count = 0;
};

namespace {

// message of the last failed tss_create on this thread (tss_last_error(NULL))
std::string& create_error() {
  static thread_local std::string e = "null context";
  return e;
}

int fail(tss_ctx* c, int code, const std::string& msg) {
  if (c) c->err = msg;
  return code;
}

// Destroys every captured verify step.  A captured step holds the addresses
// the KV binding gave it (pool pages, page table, per-sequence page-table
// offsets, the first page ids, the rotary table), so a rebind must drop them
// all; the next verify of each shape captures it again.
hipError_t drop_graphs(tss_ctx* c) {
  hipError_t first = hipSuccess;
  for (auto& g : c->graphs) {
    const hipError_t a = g.exec ? hipGraphExecDestroy(g.exec) : hipSuccess;
    const hipError_t b = g.graph ? hipGraphDestroy(g.graph) : hipSuccess;
    if (first == hipSuccess) first = a != hipSuccess ? a : b;
  }
  c->graphs.clear();
  return first;
}

int hip_fail(tss_ctx* c, hipError_t e, const char* where) {
  c->poisoned = true;
  return fail(c, TSS_EHIP, std::string(where) + ": " + hipGetErrorString(e));
}

#define HIPCHK(call, where)                      \
  do {                                           \
    hipError_t e_ = (call);                      \
    if (e_ != hipSuccess) return hip_fail(c, e_, where); \
  } while (0)

int validate_tree(const int32_t* parent, int32_t n, int32_t max_nodes) {
  if (n < 1 || n > max_nodes || n > kMaxNodes) return TSS_EINVAL;
  if (!parent) return TSS_OK;
  if (parent[0] != -1) return TSS_EINVAL;
  for (int i = 1; i < n; ++i)
    if (parent[i] < 0 || parent[i] >= i) return TSS_EINVAL;
  return TSS_OK;
}

void tree_meta(const int32_t* parent, int n, int32_t* depth, uint64_t* anc) {
  depth[0] = 0;
  anc[0] = 1ull;
  for (int i = 1; i < n; ++i) {
    const int p = parent ? parent[i] : i - 1;
    depth[i] = depth[p] + 1;
    anc[i] = anc[p] | (1ull << i);
  }
}

// Row permutation of the packed Q/K/V sections: inside each head, tile t of 16
// output rows holds dims 8t..8t+7 and hd/2+8t..hd/2+8t+7, so every rotary pair
// (j, j + hd/2) lands in one tile, 8 lanes apart.
int qkv_src_row(int n_in_section, int head_dim) {
  const int ts = n_in_section >> 4, c = n_in_section & 15;
  const int hd16 = head_dim >> 4;
  const int head = ts / hd16, t = ts % hd16;
  const int dim = c < 8 ? 8 * t + c : head_dim / 2 + 8 * t + (c - 8);
  return head * head_dim + dim;
}

// Packs rows of src [rows][K] (elements of es bytes) into 1 KiB lane-ordered
// tiles.  Output tile (r, c) for row tile r and K chunk c is written to
// dst + (r * nkc + c) * tile_stride; row_map gives the source row of packed row n.
template <typename RowMap>
void pack_tiles(uint8_t* dst, const uint8_t* src, int rows, int K, int es, size_t tile_stride, RowMap row_map,
                bool to_f16, std::atomic<bool>* ok) {
  const int KC = 64 / es, KL = KC / 4;
  const int nkc = K / KC;
  const int row_tiles = rows / 16;
  const unsigned nth = std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
  auto work = [&](int r0, int r1) {
    for (int r = r0; r < r1; ++r) {
      const uint8_t* srow[16];
      for (int i = 0; i < 16; ++i) srow[i] = src + (size_t)row_map(r * 16 + i) * K * es;
      for (int c = 0; c < nkc; ++c) {
        uint8_t* t = dst + ((size_t)r * nkc + c) * tile_stride;
        for (int l = 0; l < 64; ++l)
          copy_weights(t + l * 16, srow[l & 15] + ((size_t)c * KC + (l >> 4) * KL) * es, 16, to_f16, ok);
      }
    }
  };
  if (row_tiles < 64 || nth == 1) {
    work(0, row_tiles);
    return;
  }
  std::vector<std::thread> th;
  const int per = (row_tiles + nth - 1) / nth;
  for (unsigned i = 0; i < nth; ++i) {
    const int r0 = i * per, r1 = std::min(row_tiles, (int)(r0 + per));
    if (r0 < r1) th.emplace_back(work, r0, r1);
  }
  for (auto& t : th) t.join();
}

bool mask_ok(const uint8_t* m, int n) {
  for (int i = 0; i < n; ++i)
    if (m[i] > 1) return false;
  return true;
}

}  // namespace

extern "C" {

int tss_cfg_check(const tss_model_cfg* cfg) { return cfg_ok(cfg) ? TSS_OK : TSS_EINVAL; }

size_t tss_weights_bytes(const tss_model_cfg* cfg) { return cfg_ok(cfg) ? weight_layout(cfg).total : 0; }

int64_t tss_bf16_to_f16(const uint16_t* src, uint16_t* dst, int64_t n) {
  if (n < 0 || (n > 0 && (!src || !dst))) return -1;
  const uint16_t* tab = f16_table();
  int64_t over = 0;
  for (int64_t i = 0; i < n; ++i) {
    over += bf16_out_of_f16_range(src[i]) ? 1 : 0;
    dst[i] = tab[src[i]];
  }
  return over;
}

size_t tss_workspace_bytes(const tss_model_cfg* cfg) { return cfg_ok(cfg) ? ws_layout(cfg).total : 0; }

size_t tss_kv_bytes(const tss_model_cfg* cfg, int32_t n_seqs, int32_t max_tokens_per_seq) {
  if (!cfg_ok(cfg) || n_seqs < 1 || max_tokens_per_seq < 1) return 0;
  return kv_layout(cfg, n_seqs, max_tokens_per_seq).total;
}

int tss_validate_tree(const int32_t* parent, int32_t n_nodes, int32_t max_nodes) {
  return validate_tree(parent, n_nodes, max_nodes);
}

int tss_validate_mask(const uint8_t* mask, int32_t n_layers) {
  if (n_layers < 1 || n_layers > kMaxLayers) return TSS_EINVAL;
  if (!mask) return TSS_OK;
  return mask_ok(mask, n_layers) ? TSS_OK : TSS_EINVAL;
}

int tss_tree_meta(const int32_t* parent, int32_t n_nodes, int32_t* depth, uint64_t* anc) {
  if (!depth || !anc) return TSS_EINVAL;
  const int r = validate_tree(parent, n_nodes, kMaxNodes);
  if (r != TSS_OK) return r;
  tree_meta(parent, n_nodes, depth, anc);
  return TSS_OK;
}

const char* tss_status_string(int s) {
  switch (s) {
    case TSS_OK: return "ok";
    case TSS_EINVAL: return "invalid argument";
    case TSS_ENOSPACE: return "buffer too small";
    case TSS_ECAPACITY: return "KV capacity exceeded";
    case TSS_ESTATE: return "invalid state";
    case TSS_EHIP: return "HIP error";
    default: return "unknown status";
  }
}

const char* tss_last_error(const tss_ctx* c) { return c ? c->err.c_str() : create_error().c_str(); }

int tss_create(const tss_model_cfg* cfg, void* hip_stream, void* dev_weights, size_t weights_bytes,
               void* dev_workspace, size_t workspace_bytes, tss_ctx** out) {
  create_error() = "null context";
  if (!out) return TSS_EINVAL;
  *out = nullptr;
  if (!cfg_ok(cfg) || !dev_weights || !dev_workspace) return TSS_EINVAL;
  if (weights_bytes < weight_layout(cfg).total || workspace_bytes < ws_layout(cfg).total) return TSS_ENOSPACE;
  tss_ctx* c = new tss_ctx();
  c->cfg = *cfg;
  c->bf16 = cfg->dtype == TSS_BF16;
  c->es = elem_size(cfg);
  c->KC = 64 / c->es;
  c->Mp = round16(row_cap(cfg));
  c->stream = (hipStream_t)hip_stream;
  c->w = (uint8_t*)dev_weights;
  c->ws = c->ws_own = (uint8_t*)dev_workspace;
  c->out_ws = c->ws;
  c->wl = weight_layout(cfg);
  c->wsl = c->wsl_own = c->out_wsl = ws_layout(cfg);
  c->Mp_own = c->Mp;
  c->step.mask.reserve((size_t)kMaxSegs * cfg->n_layers);
  const char* where = "current device";
  hipError_t e = hipGetDevice(&c->device);
  if (e == hipSuccess) {
    where = "pinned step parameters";
    e = hipHostMalloc((void**)&c->sp_host, sizeof(StepParams), hipHostMallocDefault);
  }
  auto step = [&](const char* w, hipError_t r) {
    if (e == hipSuccess) {
      where = w;
      e = r;
    }
  };
  if (e == hipSuccess)
    step("mapped result buffer",
         hipHostMalloc((void**)&c->res_host, kMaxSegs * sizeof(Result), hipHostMallocMapped | hipHostMallocCoherent));
  if (e == hipSuccess) step("mapped result address", hipHostGetDevicePointer((void**)&c->res_dev_map, c->res_host, 0));
  if (e == hipSuccess)
    step("merge counters", hipMemsetAsync(c->ws + c->wsl.counters, 0, (size_t)c->wsl.n_counters * 4, c->stream));
  if (e == hipSuccess) step("stream sync", hipStreamSynchronize(c->stream));
  if (e == hipSuccess) step("attention LDS attribute", init_kernel_attributes());
  if (e == hipSuccess) step("projection LDS attribute", init_gemm_attributes());
  if (e == hipSuccess) step("timing event", hipEventCreate(&c->ev0));
  if (e == hipSuccess) step("timing event", hipEventCreate(&c->ev1));
  if (e != hipSuccess) {
    create_error() = std::string("tss_create: ") + where + ": " + hipGetErrorString(e);
    tss_destroy(c);
    return TSS_EHIP;
  }
  *out = c;
  return TSS_OK;
}

void tss_destroy(tss_ctx* c) {
  if (!c) return;
  (void)drop_graphs(c);
  if (c->cap_stream) (void)hipStreamDestroy(c->cap_stream);
  for (int i = 0; i < 2; ++i) {
    if (c->stage_ev[i]) {
      (void)hipEventSynchronize(c->stage_ev[i]);
      (void)hipEventDestroy(c->stage_ev[i]);
    }
    if (c->stage[i]) (void)hipHostFree(c->stage[i]);
  }
  if (c->sp_host) (void)hipHostFree(c->sp_host);
  if (c->res_host) (void)hipHostFree(c->res_host);
  if (c->ev0) (void)hipEventDestroy(c->ev0);
  if (c->ev1) (void)hipEventDestroy(c->ev1);
  delete c;
}

int tss_load_weights(tss_ctx* c, int32_t first, int32_t count, const void* const* host_tensors) {
  if (!c) return TSS_EINVAL;
  if (c->poisoned) return fail(c, TSS_ESTATE, "context poisoned by an earlier HIP error");
  const int L = c->cfg.n_layers, d = c->cfg.d_model, f = c->cfg.ffn_dim, v = c->cfg.vocab, es = c->es;
  const int total = 3 + 9 * L;
  if (!host_tensors || first < 0 || count < 1 || first + count > total)
    return fail(c, TSS_EINVAL, "tensor range outside the model's tensor list");
  for (int i = 0; i < count; ++i)
    if (!host_tensors[i]) return fail(c, TSS_EINVAL, "null tensor pointer");
  HIPCHK(hipStreamSynchronize(c->stream), "sync before weight load");
  if (!c->stage[0]) {
    for (int i = 0; i < 2; ++i) {
      HIPCHK(hipHostMalloc((void**)&c->stage[i], kStageBytes, hipHostMallocDefault), "pinned staging");
      HIPCHK(hipEventCreateWithFlags(&c->stage_ev[i], hipEventDisableTiming), "staging event");
      HIPCHK(hipEventRecord(c->stage_ev[i], c->stream), "staging event");
    }
  }
  // Takes the next staging buffer once its previous copy has drained.
  auto next_stage = [&](uint8_t** buf) -> hipError_t {
    const int i = c->stage_cur;
    c->stage_cur ^= 1;
    *buf = c->stage[i];
    return hipEventSynchronize(c->stage_ev[i]);
  };
  auto stage_done = [&](int used) { return hipEventRecord(c->stage_ev[used], c->stream); };
  // bf16 weights are stored as fp16 (the MFMA operand type of the mode)
  const bool to_f16 = c->bf16;
  std::atomic<bool> in_range{true};
  // raw copies: the embedding (16-bit, converted like the packed weights) and
  // the fp32 norm gains (never converted)
  auto raw = [&](size_t off, const void* src, size_t bytes, bool convert) -> hipError_t {
    for (size_t done = 0; done < bytes; done += kStageBytes) {
      const size_t n = std::min(kStageBytes, bytes - done);
      const int used = c->stage_cur;
      uint8_t* b;
      hipError_t e = next_stage(&b);
      if (e != hipSuccess) return e;
      copy_weights(b, (const uint8_t*)src + done, n, convert && to_f16, &in_range);
      e = hipMemcpyAsync(c->w + off + done, b, n, hipMemcpyHostToDevice, c->stream);
      if (e == hipSuccess) e = stage_done(used);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  };
  auto gain = [&](size_t off, const void* src) {
    std::vector<float> g(d);
    if (c->bf16) {
      const uint16_t* s = (const uint16_t*)src;
      for (int k = 0; k < d; ++k) {
        const uint32_t b = (uint32_t)s[k] << 16;
        std::memcpy(&g[k], &b, 4);
      }
    } else {
      std::memcpy(g.data(), src, (size_t)d * 4);
    }
    return raw(off, g.data(), (size_t)d * 4, false);
  };
  // Packs src [rows][K] in batches of row tiles through the staging buffers.
  // slot < 0: single-tile strips (tile (r, c) at (r * nkc + c) KiB); slot 0/1:
  // gate/up pairs (tile (r, c) at ((r * nkc + c) * 2 + slot) KiB).
  auto packed = [&](size_t off, const void* src, int rows, int K, int slot, auto row_map) -> hipError_t {
    const int nkc = K / c->KC;
    const size_t rt_bytes = (size_t)nkc * kTileBytes;
    const int per_batch = (int)std::max<size_t>(1, kStageBytes / rt_bytes);
    const int rts = rows / 16;
    for (int r0 = 0; r0 < rts; r0 += per_batch) {
      const int r1 = std::min(rts, r0 + per_batch);
      const int used = c->stage_cur;
      uint8_t* b;
      hipError_t e = next_stage(&b);
      if (e != hipSuccess) return e;
      pack_tiles(b, (const uint8_t*)src, (r1 - r0) * 16, K, es, kTileBytes,
                 [&](int n) { return row_map(r0 * 16 + n); }, to_f16, &in_range);
      if (slot < 0)
        e = hipMemcpyAsync(c->w + off + (size_t)r0 * rt_bytes, b, (size_t)(r1 - r0) * rt_bytes, hipMemcpyHostToDevice,
                           c->stream);
      else
        e = hipMemcpy2DAsync(c->w + off + ((size_t)r0 * nkc * 2 + slot) * kTileBytes, 2 * kTileBytes, b, kTileBytes,
                             kTileBytes, (size_t)(r1 - r0) * nkc, hipMemcpyHostToDevice, c->stream);
      if (e == hipSuccess) e = stage_done(used);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  };
  auto ident = [](int n) { return n; };
  for (int i = 0; i < count; ++i) {
    const int t = first + i;
    const void* src = host_tensors[i];
    hipError_t e = hipSuccess;
    if (t == 0) {
      e = raw(c->wl.embed, src, (size_t)v * d * es, true);
    } else if (t == 1 + 9 * L) {
      e = gain(c->wl.final_norm, src);
    } else if (t == 2 + 9 * L) {
      e = packed(c->wl.lm_head, src, v, d, -1, ident);
    } else {
      const int l = (t - 1) / 9, j = (t - 1) % 9;
      const LayerW& W = c->wl.layers[l];
      const int hd = c->cfg.head_dim;
      switch (j) {
        case 0: e = gain(W.attn_norm, src); break;
        case 1: case 2: case 3:
          e = packed(W.qkv + (size_t)(j - 1) * d * d * es, src, d, d, -1, [hd](int n) { return qkv_src_row(n, hd); });
          break;
        case 4: e = packed(W.o, src, d, d, -1, ident); break;
        case 5: e = gain(W.mlp_norm, src); break;
        case 6: case 7: e = packed(W.gateup, src, f, d, j - 6, ident); break;
        default: e = packed(W.down, src, d, f, -1, ident); break;
      }
    }
    if (e != hipSuccess) return hip_fail(c, e, "weight upload");
  }
  HIPCHK(hipStreamSynchronize(c->stream), "weight upload");
  if (!in_range.load())
    return fail(c, TSS_EINVAL, "a weight's magnitude exceeds 65504, the largest value of the fp16 operands");
  return TSS_OK;
}

int tss_kv_alloc(tss_ctx* c, int32_t n_seqs, int32_t max_tokens_per_seq, void* dev_pool, size_t pool_bytes,
                 const int32_t* page_order) {
  if (!c) return TSS_EINVAL;
  if (c->poisoned) return fail(c, TSS_ESTATE, "context poisoned by an earlier HIP error");
  if (n_seqs < 1 || max_tokens_per_seq < 1 || !dev_pool) return fail(c, TSS_EINVAL, "bad KV pool arguments");
  const KvLayout k = kv_layout(&c->cfg, n_seqs, max_tokens_per_seq);
  if (pool_bytes < k.total) return fail(c, TSS_ENOSPACE, "KV pool smaller than tss_kv_bytes()");
  std::vector<int32_t> pt(k.n_pages);
  if (page_order) {
    std::vector<uint8_t> seen(k.n_pages, 0);
    for (int i = 0; i < k.n_pages; ++i) {
      const int p = page_order[i];
      if (p < 0 || p >= k.n_pages || seen[p]) return fail(c, TSS_EINVAL, "page_order is not a permutation");
      seen[p] = 1;
      pt[i] = p;
    }
  } else {
    for (int i = 0; i < k.n_pages; ++i) pt[i] = i;
  }
  HIPCHK(hipStreamSynchronize(c->stream), "sync before KV bind");
  HIPCHK(drop_graphs(c), "dropping the steps captured for the previous KV binding");
  c->kv = (uint8_t*)dev_pool;
  c->kvl = k;
  c->n_seqs = n_seqs;
  c->max_tokens = max_tokens_per_seq;
  HIPCHK(hipMemcpy(c->kv + k.page_table, pt.data(), pt.size() * 4, hipMemcpyHostToDevice), "page table upload");
  c->pt_host = pt;
  HIPCHK(launch_rope_table((float2*)(c->kv + k.rope), max_tokens_per_seq, c->cfg.head_dim, c->cfg.rope_base,
                           c->stream),
         "rope table");
  HIPCHK(hipStreamSynchronize(c->stream), "rope table");
  c->n_kv.assign(n_seqs, 0);
  c->kv_len.assign(n_seqs, std::vector<int32_t>(c->cfg.n_layers, 0));
  c->mask.assign(n_seqs, std::vector<uint8_t>(c->cfg.n_layers, 0));
  return TSS_OK;
}

int tss_set_skip_mask(tss_ctx* c, int32_t seq, const uint8_t* mask) {
  if (!c) return TSS_EINVAL;
  if (seq < 0 || seq >= c->n_seqs) return fail(c, TSS_EINVAL, "unknown sequence");
  if (mask && !mask_ok(mask, c->cfg.n_layers)) return fail(c, TSS_EINVAL, "mask bytes must be 0 or 1");
  for (int l = 0; l < c->cfg.n_layers; ++l) c->mask[seq][l] = mask ? mask[l] : 0;
  return TSS_OK;
}

int tss_seq_length(tss_ctx* c, int32_t seq, int32_t* n_kv) {
  if (!c || !n_kv) return TSS_EINVAL;
  if (seq < 0 || seq >= c->n_seqs) return fail(c, TSS_EINVAL, "unknown sequence");
  *n_kv = c->n_kv[seq];
  return TSS_OK;
}

int tss_seq_truncate(tss_ctx* c, int32_t seq, int32_t n_kv) {
  if (!c) return TSS_EINVAL;
  if (seq < 0 || seq >= c->n_seqs) return fail(c, TSS_EINVAL, "unknown sequence");
  if (n_kv < 0 || n_kv > c->n_kv[seq]) return fail(c, TSS_EINVAL, "truncate can only shorten a sequence");
  c->n_kv[seq] = n_kv;
  for (auto& k : c->kv_len[seq]) k = std::min(k, n_kv);
  return TSS_OK;
}

int tss_set_launch_mode(tss_ctx* c, int32_t mode) {
  if (!c) return TSS_EINVAL;
  if (mode != TSS_LAUNCH_DIRECT && mode != TSS_LAUNCH_GRAPH) return fail(c, TSS_EINVAL, "unknown launch mode");
  c->launch_mode = mode;
  return TSS_OK;
}

int tss_profile_kernel(tss_ctx* c, int32_t kernel, int32_t layer) {
  if (!c) return TSS_EINVAL;
  if (kernel < -1 || kernel > TSS_K_COMPACT) return fail(c, TSS_EINVAL, "unknown kernel kind");
  c->prof_kind = kernel;
  c->prof_layer = layer;
  return TSS_OK;
}

int tss_profile_read(tss_ctx* c, double* total_ms, int64_t* count, int32_t reset) {
  if (!c) return TSS_EINVAL;
  if (total_ms) *total_ms = c->prof_ms;
  if (count) *count = c->prof_count;
  if (reset) {
    c->prof_ms = 0.0;
    c->prof_count = 0;
  }
  return TSS_OK;
}

}  // extern "C"

namespace {

// Binds the context's event pair to one launch when it is the profiled one.
struct ProfScope {
  tss_ctx* c;
  bool on;
  ProfScope(tss_ctx* ctx, int kind, int layer) : c(ctx) {
    on = c->prof_kind == kind && (layer < 0 || c->prof_layer == layer) && !c->prof_armed;
    if (on) launch_timing() = LaunchTiming{c->ev0, c->ev1};
  }
  void done() {
    if (on) {
      launch_timing() = LaunchTiming{};
      c->prof_armed = true;
    }
  }
  ~ProfScope() {
    if (on) launch_timing() = LaunchTiming{};
  }
};

EmbedArgs embed_args(tss_ctx* c, int start_layer = 0, const float* src_h = nullptr);


// Layer after `l` that segment i runs (n_layers = none), and the gain of the
// RMSNorm that layer (or the final norm) applies first.
int next_active(const tss_ctx* c, int i, int l) {
  const int L = c->cfg.n_layers;
  const uint8_t* m = c->step.mask.data() + (size_t)i * L;
  for (int k = l + 1; k < L; ++k)
    if (!m[k]) return k;
  return L;
}
const float* attn_gain_of(const tss_ctx* c, int layer) {
  return (const float*)(c->w + (layer < c->cfg.n_layers ? c->wl.layers[layer].attn_norm : c->wl.final_norm));
}

// Enqueues embed, the blocks that any segment of the step runs and (for
// verify) lm_head + accept (+ KV compaction) for the rows in c->sp_host and
// the segments in c->step, on stream s.  A block that every segment skips is
// not launched; inside a launched block the rows of segments that skip it
// are left untouched (their attention rows, if an item spans them, are
// computed and discarded).  Every kernel argument except the embedding
// kernel's step parameters depends only on the step's shape (segments,
// sequences, masks, node counts, compaction), not on context lengths, so a
// captured sequence of launches can be replayed for later steps of the same
// shape.
//
// start_layer > 0 resumes a step after blocks that every segment runs as the
// dense verifier does: the rows start from resume_h (the residual before
// start_layer of each local node, [n][d] fp32) instead of the embedding.
// save_prefix, when set, receives the residual of rows 0 .. prefix_rows-1
// before every block l >= 1 (at save_prefix + l * prefix_rows * d).
int enqueue_step(tss_ctx* c, bool verify, hipStream_t s, int start_layer = 0, const float* resume_h = nullptr,
                 float* save_prefix = nullptr, int prefix_rows = 0) {
  const tss_model_cfg& cf = c->cfg;
  const StepParams& sp = *c->sp_host;
  const tss_ctx::Step& st = c->step;
  const int M = sp.M, L = cf.n_layers, d = cf.d_model, f = cf.ffn_dim, H = cf.n_heads, hd = cf.head_dim;
  const int B = st.n_seqs;
  const int mt = (M + 15) / 16;
  uint8_t* ws = c->ws;
  StepParams* sp_dev = (StepParams*)(ws + c->wsl.sp);
  const int pps = c->kvl.pages_per_seq;
  const int32_t* pt_all = (const int32_t*)(c->kv + c->kvl.page_table);
  uint8_t* pages = c->kv + c->kvl.pages;
  const float2* rope = (const float2*)(c->kv + c->kvl.rope);
  c->cur_stream = s;
  c->prof_armed = false;

  int32_t pt_off[kMaxSegs] = {};
  bool one_seq = true;
  for (int i = 0; i < B; ++i) {
    pt_off[i] = st.seq[i] * pps;
    one_seq = one_seq && st.seq[i] == st.seq[0];
  }
  // with one KV sequence in the step its first page ids travel in the kernel arguments
  int32_t arg_pages[kArgPages] = {};
  const int n_arg_pages = one_seq ? std::min(pps, kArgPages) : 0;
  for (int i = 0; i < n_arg_pages; ++i) arg_pages[i] = c->pt_host[(size_t)pt_off[0] + i];

  {
    const EmbedArgs a = embed_args(c, start_layer, start_layer > 0 ? resume_h : nullptr);
    ProfScope ps(c, TSS_K_EMBED, -1);
    HIPCHK(launch_embed(c->bf16, a, s), "embed");
    ps.done();
  }

  GemmArgs base{};
  base.M = M;
  base.Mp = c->Mp;
  base.n_seqs = B;
  const bool two = act_planes(&cf) == 2;
  const size_t plane_d = two ? (size_t)c->Mp * d : 0, plane_f = two ? (size_t)c->Mp * f : 0;
  base.eps = cf.rms_eps;
  base.norm_dim = d;
  base.ss_stride = d / 16;
  base.ss_nparts = d / 16;
  base.am_stride = cf.vocab / 16;
  base.ksplit = 1;
  base.wide_wgs = 0;
  base.sp = sp_dev;
  base.row_on[0] = base.row_on[1] = ~0ull;

  for (int l = start_layer; l < L; ++l) {
    if (save_prefix && l > 0)
      HIPCHK(hipMemcpyAsync(save_prefix + (size_t)l * prefix_rows * d, ws + c->wsl.h, (size_t)prefix_rows * d * 4,
                            hipMemcpyDeviceToDevice, s),
             "prefix save");
    // rows and segments that run block l; attention items: per KV sequence
    // (a run of segments with the same sequence), the rows from its first to
    // its last segment that runs the block, cut into pieces of 64 rows
    uint64_t row_on[kMaxRows / 64] = {0, 0};
    AttnArgs at{};
    int n_act = 0, max_tiles = 1;
    for (int u0 = 0; u0 < B;) {
      int u1 = u0 + 1;
      while (u1 < B && st.seq[u1] == st.seq[u0]) ++u1;
      int lo = -1, hi = -1;
      for (int i = u0; i < u1; ++i) {
        if (st.mask[(size_t)i * L + l]) continue;
        const int r0 = sp.seq_row0[i], r1 = sp.seq_row0[i + 1];
        for (int r = r0; r < r1; ++r) row_on[r >> 6] |= 1ull << (r & 63);
        if (lo < 0) lo = r0;
        hi = r1;
      }
      for (int r = lo; lo >= 0 && r < hi; r += 4 * 16) {
        if (n_act == kAttnMaxItems) return fail(c, TSS_EINVAL, "too many attention items in one step");
        const int rows = std::min(64, hi - r);
        const int last_seg = sp.row_seq[r + rows - 1];
        at.item_row0[n_act] = r;
        at.item_rows[n_act] = rows;
        at.item_seg[n_act] = sp.row_seq[r];
        at.item_slots[n_act] = sp.seg_slot0[last_seg] + sp.seq_row0[last_seg + 1] - sp.seq_row0[last_seg];
        max_tiles = std::max(max_tiles, (rows + 15) / 16);
        ++n_act;
      }
      u0 = u1;
    }
    if (n_act == 0) continue;  // every segment skips this block
    const LayerW& W = c->wl.layers[l];
    GemmArgs lb = base;
    lb.row_on[0] = row_on[0];
    lb.row_on[1] = row_on[1];
    {  // RMSNorm + QKV + RoPE + KV append
      GemmArgs a = lb;
      a.w = c->w + W.qkv;
      a.x = ws + c->wsl.xa;
      a.x_plane = plane_d;
      a.K = d;
      a.N = 3 * d;
      a.nkc = d / c->KC;
      a.ss_in = (const float*)(ws + c->wsl.ss_a);
      a.q = (float*)(ws + c->wsl.q);
      a.kv_pages = pages;
      a.page_table = pt_all;
      std::memcpy(a.pt_off, pt_off, sizeof(pt_off));
      a.n_arg_pages = n_arg_pages;
      std::memcpy(a.pages, arg_pages, sizeof(arg_pages));
      a.rope = rope;
      a.layer = l;
      a.n_pages_pool = c->kvl.n_pages;
      a.n_heads = H;
      a.head_dim = hd;
      a.d = d;
      ProfScope ps(c, TSS_K_QKV, l);
      HIPCHK(launch_gemm(c->bf16, EPI_QKV, mt, gemm_tiles(EPI_QKV, mt, a.N), a, s), "qkv gemm");
      ps.done();
    }
    {  // tree attention
      AttnArgs& a = at;
      a.q = (const float*)(ws + c->wsl.q);
      a.kv_pages = pages;
      a.page_table = pt_all;
      a.sp = sp_dev;
      a.o = ws + c->wsl.o;
      a.o_plane = plane_d;
      std::memcpy(a.pt_off, pt_off, sizeof(pt_off));
      a.n_arg_pages = n_arg_pages;
      std::memcpy(a.pages, arg_pages, sizeof(arg_pages));
      a.part_o = (float*)(ws + c->wsl.part_o);
      a.part_ml = (float*)(ws + c->wsl.part_ml);
      a.counters = (int*)(ws + c->wsl.counters);
      a.split_out = (int32_t*)(ws + c->wsl.attn_split);
      if (!one_seq && n_act > 1) {
        a.groups = attn_batch_groups(H, n_act, pps);
        a.pages_per_wg = kAttnPagesPerWG;
      } else {
        a.groups = attn_groups(H, n_act);
        a.pages_per_wg = 0;
      }
      a.defer_merge = max_tiles >= 2;
      a.layer = l;
      a.n_pages_pool = c->kvl.n_pages;
      a.n_heads = H;
      a.d = d;
      a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)hd));
      ProfScope ps(c, TSS_K_ATTN, l);
      HIPCHK(launch_attn(c->bf16, hd, max_tiles, n_act, a, s), "attention");
      ps.done();
    }
    {  // O projection + residual; next norm input (this block's MLP norm)
      GemmArgs a = lb;
      a.w = c->w + W.o;
      a.x = ws + c->wsl.o;
      a.x_plane = plane_d;
      a.K = d;
      a.N = d;
      a.nkc = d / c->KC;
      a.h = (float*)(ws + c->wsl.h);
      a.xn = ws + c->wsl.xm;
      a.xn_plane = plane_d;
      for (int i = 0; i < kMaxSegs; ++i) a.g_next[i] = (const float*)(c->w + W.mlp_norm);
      a.ss_out = (float*)(ws + c->wsl.ss_m);
      ProfScope ps(c, TSS_K_OPROJ, l);
      a.ksplit = gemm_ksplit(EPI_RESID, mt, a.N, a.nkc);
      a.kpart = (float*)(ws + c->wsl.kpart);
      a.kcount = (int*)(ws + c->wsl.kcount);
      HIPCHK(launch_gemm(c->bf16, EPI_RESID, mt, gemm_tiles(EPI_RESID, mt, a.N), a, s), "o gemm");
      ps.done();
    }
    {  // RMSNorm + gate/up + SwiGLU
      GemmArgs a = lb;
      a.w = c->w + W.gateup;
      a.x = ws + c->wsl.xm;
      a.x_plane = plane_d;
      a.K = d;
      a.N = 2 * f;
      a.nkc = d / c->KC;
      a.ss_in = (const float*)(ws + c->wsl.ss_m);
      a.act = ws + c->wsl.act;
      a.act_plane = plane_f;
      a.wide_wgs = gemm_wide_wgs(EPI_SWIGLU, mt, a.N);
      ProfScope ps(c, TSS_K_GATEUP, l);
      HIPCHK(launch_gemm(c->bf16, EPI_SWIGLU, mt, gemm_tiles(EPI_SWIGLU, mt, a.N), a, s), "gate/up gemm");
      ps.done();
    }
    {  // down projection + residual; next norm input (each sequence's next block, or the final norm)
      GemmArgs a = lb;
      a.w = c->w + W.down;
      a.x = ws + c->wsl.act;
      a.x_plane = plane_f;
      a.K = f;
      a.N = d;
      a.nkc = f / c->KC;
      a.h = (float*)(ws + c->wsl.h);
      a.xn = ws + c->wsl.xa;
      a.xn_plane = plane_d;
      for (int i = 0; i < kMaxSegs; ++i) a.g_next[i] = attn_gain_of(c, i < B ? next_active(c, i, l) : L);
      a.ss_out = (float*)(ws + c->wsl.ss_a);
      ProfScope ps(c, TSS_K_DOWN, l);
      a.ksplit = gemm_ksplit(EPI_RESID, mt, a.N, a.nkc);
      a.kpart = (float*)(ws + c->wsl.kpart);
      a.kcount = (int*)(ws + c->wsl.kcount);
      HIPCHK(launch_gemm(c->bf16, EPI_RESID, mt, gemm_tiles(EPI_RESID, mt, a.N), a, s), "down gemm");
      ps.done();
    }
  }

  if (verify) {
    {  // final norm + lm_head + per-strip argmax
      GemmArgs a = base;
      a.w = c->w + c->wl.lm_head;
      a.x = ws + c->wsl.xa;
      a.x_plane = plane_d;
      a.K = d;
      a.N = cf.vocab;
      a.nkc = d / c->KC;
      a.ss_in = (const float*)(ws + c->wsl.ss_a);
      a.logits = (float*)(ws + c->wsl.logits);
      a.am_val = (float*)(ws + c->wsl.am_val);
      a.am_idx = (int32_t*)(ws + c->wsl.am_idx);
      ProfScope ps(c, TSS_K_LMHEAD, -1);
      HIPCHK(launch_gemm(c->bf16, EPI_LOGITS, mt, gemm_tiles(EPI_LOGITS, mt, a.N), a, s), "lm_head gemm");
      ps.done();
    }
    {
      AcceptArgs a{};
      a.am_val = (const float*)(ws + c->wsl.am_val);
      a.am_idx = (const int32_t*)(ws + c->wsl.am_idx);
      a.nparts = cf.vocab / 16;
      a.M = M;
      a.am_stride = cf.vocab / 16;
      a.sp = sp_dev;
      a.greedy = (int32_t*)(ws + c->wsl.greedy);
      a.count = (int*)(ws + c->wsl.acount);
      a.result = (Result*)(ws + c->wsl.result);
      a.result_host = c->res_dev_map;
      ProfScope ps(c, TSS_K_ACCEPT, -1);
      HIPCHK(launch_accept(a, s), "accept");
      ps.done();
    }
    CompactArgs a{};
    int nz = 0;
    for (int i = 0; i < B; ++i) {
      if (!st.compact[i]) continue;
      a.seq[nz] = i;
      a.pt_off[nz] = pt_off[i];
      for (int l = 0; l < L; ++l)
        if (!st.mask[(size_t)i * L + l]) a.lay_on[nz][l >> 6] |= 1ull << (l & 63);
      ++nz;
    }
    if (nz > 0) {
      a.kv_pages = pages;
      a.page_table = pt_all;
      a.sp = sp_dev;
      a.result = (const Result*)(ws + c->wsl.result);
      a.n_layers = L;
      a.n_pages_pool = c->kvl.n_pages;
      a.n_heads = H;
      a.head_dim = hd;
      ProfScope ps(c, TSS_K_COMPACT, -1);
      HIPCHK(launch_compact(c->bf16, nz, a, s), "kv compaction");
      ps.done();
    }
  }
  return TSS_OK;
}

// Waits for the step and collects the profiled launch's event times.  The
// step's outputs (logits, greedy tokens, split report) are in the workspace
// it ran on, whether it was enqueued now or replayed from a captured graph.
int finish_step(tss_ctx* c) {
  HIPCHK(hipStreamSynchronize(c->stream), "step");
  c->out_ws = c->ws;
  c->out_wsl = c->wsl;
  if (c->prof_armed) {
    float ms = 0.f;
    HIPCHK(hipEventElapsedTime(&ms, c->ev0, c->ev1), "event timing");
    c->prof_ms += ms;
    c->prof_count += 1;
    c->prof_armed = false;
  }
  return TSS_OK;
}

int run_step(tss_ctx* c, bool verify, int start_layer = 0, const float* resume_h = nullptr,
             float* save_prefix = nullptr, int prefix_rows = 0) {
  const int r = enqueue_step(c, verify, c->stream, start_layer, resume_h, save_prefix, prefix_rows);
  if (r) return r;
  return finish_step(c);
}

// The embedding kernel's arguments for the step in c->sp_host (the only
// per-step arguments of a verify); a resumed step starts at start_layer from
// the saved residual rows src_h.
EmbedArgs embed_args(tss_ctx* c, int start_layer, const float* src_h) {
  const tss_model_cfg& cf = c->cfg;
  const StepParams& sp = *c->sp_host;
  EmbedArgs a{};
  a.embed = c->w + c->wl.embed;
  a.sp = sp;
  a.sp_dev = (StepParams*)(c->ws + c->wsl.sp);
  for (int i = 0; i < kMaxSegs; ++i)
    a.gain[i] = attn_gain_of(c, i < c->step.n_seqs ? next_active(c, i, start_layer - 1) : 0);
  a.src_h = src_h;
  a.h = (float*)(c->ws + c->wsl.h);
  a.xn = c->ws + c->wsl.xa;
  a.xn_plane = act_planes(&cf) == 2 ? (size_t)c->Mp * cf.d_model : 0;
  a.ss_out = (float*)(c->ws + c->wsl.ss_a);
  a.ss_stride = cf.d_model / 16;
  a.d = cf.d_model;
  a.M = sp.M;
  a.attn_split = (int32_t*)(c->ws + c->wsl.attn_split);
  a.counters = (int32_t*)(c->ws + c->wsl.counters);
  a.n_counters = c->wsl.n_counters;
  return a;
}

// A verify step from the graph cache: captured on first use of its shape,
// then replayed with the embedding kernel's step parameters updated.
int run_verify_graph(tss_ctx* c) {
  const StepParams& sp = *c->sp_host;
  const tss_ctx::Step& st = c->step;
  std::string key;
  key.reserve(64 + st.mask.size());
  auto put = [&](int v) { key.append((const char*)&v, sizeof(v)); };
  put(st.n_seqs);
  for (int i = 0; i < st.n_seqs; ++i) {
    put(st.seq[i]);
    put(sp.seq_row0[i + 1] - sp.seq_row0[i]);
    put(st.compact[i]);
  }
  key.append((const char*)st.mask.data(), st.mask.size());
  tss_ctx::GraphEntry* g = nullptr;
  for (auto& e : c->graphs)
    if (e.key == key) g = &e;
  if (!g) {
    constexpr size_t kMaxGraphs = 32;
    if (c->graphs.size() >= kMaxGraphs) {  // drop the least recently used
      size_t old = 0;
      for (size_t i = 1; i < c->graphs.size(); ++i)
        if (c->graphs[i].last_use < c->graphs[old].last_use) old = i;
      HIPCHK(hipGraphExecDestroy(c->graphs[old].exec), "graph destroy");
      HIPCHK(hipGraphDestroy(c->graphs[old].graph), "graph destroy");
      c->graphs.erase(c->graphs.begin() + old);
    }
    if (!c->cap_stream) HIPCHK(hipStreamCreateWithFlags(&c->cap_stream, hipStreamNonBlocking), "capture stream");
    tss_ctx::GraphEntry e;
    e.key = key;
    c->prof_armed = false;
    HIPCHK(hipStreamBeginCapture(c->cap_stream, hipStreamCaptureModeThreadLocal), "begin capture");
    const int r = enqueue_step(c, true, c->cap_stream);
    hipGraph_t graph = nullptr;
    const hipError_t ce = hipStreamEndCapture(c->cap_stream, &graph);
    if (r) {
      if (graph) (void)hipGraphDestroy(graph);
      return r;
    }
    HIPCHK(ce, "end capture");
    e.graph = graph;
    c->prof_armed = false;
    HIPCHK(hipGraphInstantiate(&e.exec, graph, nullptr, nullptr, 0), "graph instantiate");
    size_t n = 0;
    HIPCHK(hipGraphGetNodes(graph, nullptr, &n), "graph nodes");
    std::vector<hipGraphNode_t> nodes(n);
    HIPCHK(hipGraphGetNodes(graph, nodes.data(), &n), "graph nodes");
    const void* ek = embed_kernel(c->bf16);
    for (auto node : nodes) {
      hipGraphNodeType t;
      HIPCHK(hipGraphNodeGetType(node, &t), "graph node type");
      if (t != hipGraphNodeTypeKernel) continue;
      hipKernelNodeParams kp{};
      HIPCHK(hipGraphKernelNodeGetParams(node, &kp), "graph node params");
      if (kp.func == ek) {
        e.embed_node = node;
        e.embed_params = kp;
        break;
      }
    }
    if (!e.embed_node) {
      (void)hipGraphExecDestroy(e.exec);
      (void)hipGraphDestroy(graph);
      return fail(c, TSS_EHIP, "captured step has no embedding launch");
    }
    c->graphs.push_back(e);
    g = &c->graphs.back();
  }
  g->last_use = ++c->graph_clock;
  EmbedArgs a = embed_args(c);
  void* kargs[1] = {&a};
  hipKernelNodeParams kp = g->embed_params;
  kp.kernelParams = kargs;
  kp.extra = nullptr;
  HIPCHK(hipGraphExecKernelNodeSetParams(g->exec, g->embed_node, &kp), "graph update");
  HIPCHK(hipGraphLaunch(g->exec, c->stream), "graph launch");
  return finish_step(c);
}

int check_ready(tss_ctx* c, int seq) {
  if (c->poisoned) return fail(c, TSS_ESTATE, "context poisoned by an earlier HIP error");
  if (!c->kv) return fail(c, TSS_ESTATE, "no KV pool bound (tss_kv_alloc)");
  if (seq < 0 || seq >= c->n_seqs) return fail(c, TSS_EINVAL, "unknown sequence");
  return TSS_OK;
}

// The verify of a batch of sequences (tss_verify is a batch of one).  Every
// check runs before anything is enqueued; sequence state changes only after
// the step succeeded.
int verify_batch(tss_ctx* c, int32_t n_seqs, const int32_t* seq_ids, const int32_t* node_offsets,
                 const int32_t* tokens, const int32_t* parents, const uint8_t* masks, uint32_t flags,
                 int32_t* accept_len, int32_t* next_token) {
  if (c->poisoned) return fail(c, TSS_ESTATE, "context poisoned by an earlier HIP error");
  if (!c->kv) return fail(c, TSS_ESTATE, "no KV pool bound (tss_kv_alloc)");
  if (n_seqs < 1 || n_seqs > c->cfg.max_batch) return fail(c, TSS_EINVAL, "n_seqs outside [1, max_batch]");
  if (!seq_ids || !node_offsets || !tokens || !accept_len || !next_token) return fail(c, TSS_EINVAL, "null argument");
  if (flags & ~(uint32_t)TSS_COMMIT) return fail(c, TSS_EINVAL, "unknown flag");
  const int L = c->cfg.n_layers;
  if (node_offsets[0] != 0) return fail(c, TSS_EINVAL, "node_offsets[0] must be 0");
  for (int i = 0; i < n_seqs; ++i) {
    const int sq = seq_ids[i];
    if (sq < 0 || sq >= c->n_seqs) return fail(c, TSS_EINVAL, "unknown sequence");
    for (int j = 0; j < i; ++j)
      if (seq_ids[j] == sq) return fail(c, TSS_EINVAL, "a sequence appears twice in one batch");
    const int n = node_offsets[i + 1] - node_offsets[i];
    if (validate_tree(parents ? parents + node_offsets[i] : nullptr, n, c->cfg.max_nodes) != TSS_OK)
      return fail(c, TSS_EINVAL, "invalid draft tree (n_nodes, parent[0] = -1, 0 <= parent[i] < i)");
  }
  const int M = node_offsets[n_seqs];
  if (M > row_cap(&c->cfg))
    return fail(c, TSS_EINVAL, "the batch's nodes exceed the step's row capacity");
  if (masks && !mask_ok(masks, n_seqs * L)) return fail(c, TSS_EINVAL, "mask bytes must be 0 or 1");
  for (int r = 0; r < M; ++r)
    if (tokens[r] < 0 || tokens[r] >= c->cfg.vocab) return fail(c, TSS_EINVAL, "token outside [0, vocab)");
  for (int i = 0; i < n_seqs; ++i) {
    const int sq = seq_ids[i];
    const int n = node_offsets[i + 1] - node_offsets[i];
    if (c->n_kv[sq] + n > c->max_tokens) return fail(c, TSS_ECAPACITY, "verify exceeds the sequence's KV capacity");
    const uint8_t* m = masks ? masks + (size_t)i * L : c->mask[sq].data();
    for (int l = 0; l < L; ++l)
      if (!m[l] && c->kv_len[sq][l] != c->n_kv[sq])
        return fail(c, TSS_ESTATE, "an active layer lacks K/V for the committed context");
  }

  const bool commit = flags & TSS_COMMIT;
  StepParams& sp = *c->sp_host;
  std::memset(&sp, 0, sizeof(sp));
  tss_ctx::Step& st = c->step;
  st.n_seqs = n_seqs;
  st.mask.resize((size_t)n_seqs * L);
  sp.M = M;
  sp.n_seqs = n_seqs;
  for (int i = 0; i < n_seqs; ++i) {
    const int sq = seq_ids[i], r0 = node_offsets[i], n = node_offsets[i + 1] - r0;
    st.seq[i] = sq;
    std::memcpy(st.mask.data() + (size_t)i * L, masks ? masks + (size_t)i * L : c->mask[sq].data(), L);
    sp.seq_row0[i] = r0;
    sp.seq_nkv[i] = c->n_kv[sq];
    int32_t depth[kMaxNodes];
    uint64_t anc[kMaxNodes];
    const int32_t* par = parents ? parents + r0 : nullptr;
    tree_meta(par, n, depth, anc);
    bool chain = true;
    for (int j = 0; j < n; ++j) {
      const int p = par ? par[j] : j - 1;
      if (j > 0 && p != j - 1) chain = false;
      sp.tok[r0 + j] = tokens[r0 + j];
      sp.parent[r0 + j] = (int8_t)p;
      sp.depth[r0 + j] = (uint8_t)depth[j];
      sp.anc[r0 + j] = anc[j];
      sp.row_seq[r0 + j] = (uint8_t)i;
      sp.row_slot0[r0 + j] = sp.seg_slot0[i];
    }
    st.compact[i] = commit && !chain;
  }
  sp.seq_row0[n_seqs] = M;
  // event timing of one launch needs direct launches (events recorded inside a
  // captured graph cannot be timed)
  const bool graph = c->launch_mode == TSS_LAUNCH_GRAPH && c->prof_kind < 0 && !c->direct_only;
  const int r = graph ? run_verify_graph(c) : run_step(c, true);
  if (r) return r;
  c->last_M = M;
  c->last_results = n_seqs;
  for (int i = 0; i < n_seqs; ++i) {
    const int sq = seq_ids[i];
    accept_len[i] = c->res_host[i].accept_len;
    next_token[i] = c->res_host[i].next_token;
    if (commit) {
      c->n_kv[sq] += c->res_host[i].accept_len + 1;
      const uint8_t* m = st.mask.data() + (size_t)i * L;
      for (int l = 0; l < L; ++l)
        if (!m[l]) c->kv_len[sq][l] = c->n_kv[sq];
    }
  }
  return TSS_OK;
}

// One draft tree of one sequence verified under many skip masks (dry runs):
// consecutive masks are packed into steps of several segments that share the
// sequence's context (each segment takes its own draft slots after it), so a
// step reads each launched block's weights and each context page once for
// all of its masks.  Direct launches: sweep steps rarely repeat a shape, and
// capturing each would cost more than it saves and evict the decode steps'
// graphs.
//
// With a prefix buffer, the shared prefix is reused as well: a mask runs
// every block before its first skipped one exactly as the dense verifier
// does, so the masks are ordered by their first skipped block (latest first),
// one dense pass saves every node's residual before every block, and each
// step starts at the earliest first-skipped block among its masks from that
// saved residual.  The dense pass itself answers the dense masks.  It is
// taken only when the blocks it saves exceed the blocks it costs.
size_t sweep_prefix_bytes(const tss_model_cfg* cf, int n) {
  return (size_t)cf->n_layers * n * cf->d_model * 4;
}

int verify_sweep(tss_ctx* c, int32_t seq, const int32_t* tokens, const int32_t* parent, int32_t n,
                 int32_t n_masks, const uint8_t* masks, int32_t* accept_len, int32_t* next_token, int32_t* greedy,
                 void* prefix, size_t prefix_bytes) {
  int r = check_ready(c, seq);
  if (r) return r;
  if (!tokens || !masks || !accept_len || !next_token) return fail(c, TSS_EINVAL, "null argument");
  if (n_masks < 1) return fail(c, TSS_EINVAL, "n_masks must be at least 1");
  if (validate_tree(parent, n, c->cfg.max_nodes) != TSS_OK)
    return fail(c, TSS_EINVAL, "invalid draft tree (n_nodes, parent[0] = -1, 0 <= parent[i] < i)");
  for (int j = 0; j < n; ++j)
    if (tokens[j] < 0 || tokens[j] >= c->cfg.vocab) return fail(c, TSS_EINVAL, "token outside [0, vocab)");
  const int L = c->cfg.n_layers;
  if (!mask_ok(masks, n_masks * L)) return fail(c, TSS_EINVAL, "mask bytes must be 0 or 1");
  if (prefix && prefix_bytes < sweep_prefix_bytes(&c->cfg, n))
    return fail(c, TSS_ENOSPACE, "prefix buffer smaller than tss_sweep_prefix_bytes");
  if (c->n_kv[seq] + n > c->max_tokens) return fail(c, TSS_ECAPACITY, "verify exceeds the sequence's KV capacity");
  for (int k = 0; k < n_masks; ++k)
    for (int l = 0; l < L; ++l)
      if (!masks[(size_t)k * L + l] && c->kv_len[seq][l] != c->n_kv[seq])
        return fail(c, TSS_ESTATE, "an active layer lacks K/V for the committed context");
  // masks per step: segment limit, row capacity, draft slots left in the sequence
  const int per_step = std::min({kMaxSegs, row_cap(&c->cfg) / n, (c->max_tokens - c->n_kv[seq]) / n});
  int32_t depth[kMaxNodes];
  uint64_t anc[kMaxNodes];
  tree_meta(parent, n, depth, anc);

  // first skipped block of each mask (L: dense), and the order of the masks
  std::vector<int> first(n_masks, L), ord(n_masks);
  for (int k = 0; k < n_masks; ++k) {
    ord[k] = k;
    for (int l = 0; l < L; ++l)
      if (masks[(size_t)k * L + l]) {
        first[k] = l;
        break;
      }
  }
  int n_dense = 0;
  bool reuse = false;
  if (prefix) {
    std::stable_sort(ord.begin(), ord.end(), [&](int x, int y) { return first[x] > first[y]; });
    while (n_dense < n_masks && first[ord[n_dense]] == L) ++n_dense;
    long saved = 0;
    for (int k0 = n_dense; k0 < n_masks; k0 += per_step) saved += first[ord[std::min(k0 + per_step, n_masks) - 1]];
    reuse = saved > L;
  }
  float* pre = (float*)prefix;
  const int d = c->cfg.d_model;

  tss_ctx::Step& st = c->step;
  auto fill = [&](int P) {  // the step's parameters for P segments of the tree
    StepParams& sp = *c->sp_host;
    std::memset(&sp, 0, sizeof(sp));
    sp.M = P * n;
    sp.n_seqs = P;
    st.n_seqs = P;
    for (int i = 0; i < P; ++i) {
      const int r0 = i * n;
      st.seq[i] = seq;
      st.compact[i] = false;
      sp.seq_row0[i] = r0;
      sp.seq_nkv[i] = c->n_kv[seq];
      sp.seg_slot0[i] = (uint8_t)r0;
      for (int j = 0; j < n; ++j) {
        sp.tok[r0 + j] = tokens[j];
        sp.parent[r0 + j] = (int8_t)(parent ? parent[j] : j - 1);
        sp.depth[r0 + j] = (uint8_t)depth[j];
        sp.anc[r0 + j] = anc[j];
        sp.row_seq[r0 + j] = (uint8_t)i;
        sp.row_slot0[r0 + j] = (uint8_t)r0;
      }
    }
    sp.seq_row0[P] = P * n;
  };
  auto collect = [&](const int* ks, int P) -> int {  // results of mask ks[i] from segment i
    c->last_M = P * n;
    c->last_results = P;
    for (int i = 0; i < P; ++i) {
      accept_len[ks[i]] = c->res_host[i].accept_len;
      next_token[ks[i]] = c->res_host[i].next_token;
    }
    if (greedy) {
      std::vector<int32_t> g((size_t)P * n);
      HIPCHK(hipMemcpy(g.data(), c->ws + c->wsl.greedy, (size_t)P * n * 4, hipMemcpyDeviceToHost), "greedy copy");
      for (int i = 0; i < P; ++i) std::memcpy(greedy + (size_t)ks[i] * n, g.data() + (size_t)i * n, (size_t)n * 4);
    }
    return TSS_OK;
  };

  int k0 = 0;
  if (reuse) {
    // the dense pass: saves the prefix, answers the dense masks
    fill(1);
    st.mask.assign(L, 0);
    r = run_step(c, true, 0, nullptr, pre, n);
    if (r) return r;
    for (int k = 0; k < n_dense; ++k) {
      r = collect(&ord[k], 1);
      if (r) return r;
    }
    k0 = n_dense;
  }
  for (; k0 < n_masks; k0 += per_step) {
    const int P = std::min(per_step, n_masks - k0);
    fill(P);
    st.mask.resize((size_t)P * L);
    for (int i = 0; i < P; ++i) std::memcpy(st.mask.data() + (size_t)i * L, masks + (size_t)ord[k0 + i] * L, L);
    const int start = reuse ? first[ord[k0 + P - 1]] : 0;  // the earliest first skip of the step
    r = run_step(c, true, start, start > 0 ? pre + (size_t)start * n * d : nullptr);
    if (r) return r;
    r = collect(&ord[k0], P);
    if (r) return r;
  }
  return TSS_OK;
}

}  // namespace

extern "C" {

size_t tss_sweep_prefix_bytes(const tss_model_cfg* cfg, int32_t n_nodes) {
  return cfg_ok(cfg) && n_nodes >= 1 && n_nodes <= cfg->max_nodes ? sweep_prefix_bytes(cfg, n_nodes) : 0;
}

int tss_verify_sweep(tss_ctx* c, int32_t seq, const int32_t* draft_tokens, const int32_t* tree_parent,
                     int32_t n_nodes, int32_t n_masks, const uint8_t* skip_masks, int32_t* accept_len,
                     int32_t* next_token, int32_t* greedy, void* dev_prefix, size_t prefix_bytes) {
  if (!c) return TSS_EINVAL;
  return verify_sweep(c, seq, draft_tokens, tree_parent, n_nodes, n_masks, skip_masks, accept_len, next_token,
                      greedy, dev_prefix, prefix_bytes);
}

int tss_prefill(tss_ctx* c, int32_t seq, const int32_t* tokens, int32_t n) {
  if (!c) return TSS_EINVAL;
  int r = check_ready(c, seq);
  if (r) return r;
  if (n < 0 || (n > 0 && !tokens)) return fail(c, TSS_EINVAL, "bad token array");
  for (int i = 0; i < n; ++i)
    if (tokens[i] < 0 || tokens[i] >= c->cfg.vocab) return fail(c, TSS_EINVAL, "token outside [0, vocab)");
  if (c->n_kv[seq] + n > c->max_tokens) return fail(c, TSS_ECAPACITY, "prefill exceeds the sequence's KV capacity");
  const int L = c->cfg.n_layers;
  for (int l = 0; l < L; ++l)
    if (!c->mask[seq][l] && c->kv_len[seq][l] != c->n_kv[seq])
      return fail(c, TSS_ESTATE, "an active layer lacks K/V for the committed context");
  // chunks as large as the step's rows allow (a chain of at most 64 nodes)
  const int chunk = std::min(kMaxNodes, row_cap(&c->cfg));
  tss_ctx::Step& st = c->step;
  st.n_seqs = 1;
  st.seq[0] = seq;
  st.compact[0] = false;
  st.mask.assign(c->mask[seq].begin(), c->mask[seq].end());
  for (int done = 0; done < n; done += chunk) {
    const int M = std::min(chunk, n - done);
    StepParams& sp = *c->sp_host;
    std::memset(&sp, 0, sizeof(sp));
    sp.M = M;
    sp.n_seqs = 1;
    sp.seq_row0[1] = M;
    sp.seq_nkv[0] = c->n_kv[seq];
    for (int i = 0; i < M; ++i) {
      sp.tok[i] = tokens[done + i];
      sp.parent[i] = (int8_t)(i - 1);
      sp.depth[i] = (uint8_t)i;
      sp.anc[i] = (i == 63) ? ~0ull : ((1ull << (i + 1)) - 1);
    }
    r = run_step(c, false);
    if (r) return r;
    c->n_kv[seq] += M;
    for (int l = 0; l < L; ++l)
      if (!c->mask[seq][l]) c->kv_len[seq][l] = c->n_kv[seq];
  }
  return TSS_OK;
}

int tss_verify(tss_ctx* c, int32_t seq, const int32_t* draft_tokens, const int32_t* tree_parent, int32_t n_nodes,
               const uint8_t* skip_mask, uint32_t flags, int32_t* accept_len, int32_t* next_token) {
  if (!c) return TSS_EINVAL;
  const int r = check_ready(c, seq);
  if (r) return r;
  const int32_t offs[2] = {0, n_nodes};
  return verify_batch(c, 1, &seq, offs, draft_tokens, tree_parent, skip_mask, flags, accept_len, next_token);
}

size_t tss_static_workspace_bytes(const tss_model_cfg* cfg) {
  if (!cfg_ok(cfg)) return 0;
  tss_model_cfg one = *cfg;
  one.max_batch = 1;
  return ws_layout(&one).total;
}

int tss_verify_batch(tss_ctx* c, int32_t n_seqs, const int32_t* seq_ids, const int32_t* node_offsets,
                     const int32_t* draft_tokens, const int32_t* tree_parents, const uint8_t* skip_masks,
                     uint32_t flags, int32_t* accept_len, int32_t* next_token) {
  if (!c) return TSS_EINVAL;
  return verify_batch(c, n_seqs, seq_ids, node_offsets, draft_tokens, tree_parents, skip_masks, flags, accept_len,
                      next_token);
}

int tss_get_logits(tss_ctx* c, float* host_dst, int32_t n_nodes) {
  if (!c || !host_dst) return TSS_EINVAL;
  if (c->poisoned) return fail(c, TSS_ESTATE, "context poisoned by an earlier HIP error");
  if (n_nodes < 1 || n_nodes > c->last_M) return fail(c, TSS_EINVAL, "n_nodes exceeds the last verify's nodes");
  HIPCHK(hipStreamSynchronize(c->stream), "sync");
  HIPCHK(hipMemcpy(host_dst, c->out_ws + c->out_wsl.logits, (size_t)n_nodes * c->cfg.vocab * 4,
                   hipMemcpyDeviceToHost),
         "logits copy");
  return TSS_OK;
}

int tss_get_path(tss_ctx* c, int32_t index, int32_t* path_nodes, int32_t* path_len) {
  if (!c || !path_nodes || !path_len) return TSS_EINVAL;
  if (c->poisoned) return fail(c, TSS_ESTATE, "context poisoned by an earlier HIP error");
  if (index < 0 || index >= c->last_results) return fail(c, TSS_EINVAL, "no such result in the last verify");
  const Result& r = c->res_host[index];
  *path_len = r.path_len;
  for (int i = 0; i < r.path_len; ++i) path_nodes[i] = r.path[i];
  return TSS_OK;
}

int tss_get_logits_device(tss_ctx* c, float* dev_dst, int32_t n_nodes) {
  if (!c || !dev_dst) return TSS_EINVAL;
  if (c->poisoned) return fail(c, TSS_ESTATE, "context poisoned by an earlier HIP error");
  if (n_nodes < 1 || n_nodes > c->last_M) return fail(c, TSS_EINVAL, "n_nodes exceeds the last verify's nodes");
  HIPCHK(hipMemcpyAsync(dev_dst, c->out_ws + c->out_wsl.logits, (size_t)n_nodes * c->cfg.vocab * 4,
                        hipMemcpyDeviceToDevice,
                        c->stream),
         "logits copy");
  return TSS_OK;
}

int tss_get_attn_split(tss_ctx* c, int32_t* n_items, int32_t* groups, int32_t* rows) {
  if (!c || !n_items || !groups || !rows) return TSS_EINVAL;
  if (c->poisoned) return fail(c, TSS_ESTATE, "context poisoned by an earlier HIP error");
  int32_t rep[2 * kAttnMaxItems + 1];
  HIPCHK(hipStreamSynchronize(c->stream), "sync");
  HIPCHK(hipMemcpy(rep, c->out_ws + c->out_wsl.attn_split, sizeof(rep), hipMemcpyDeviceToHost), "split copy");
  const int n = std::max(0, std::min(rep[2 * kAttnMaxItems], kAttnMaxItems));
  *n_items = n;
  for (int i = 0; i < n; ++i) {
    groups[i] = rep[i];
    rows[i] = rep[kAttnMaxItems + i];
  }
  return TSS_OK;
}

int tss_check_kv(tss_ctx* c) {
  if (!c) return TSS_EINVAL;
  if (c->poisoned) return fail(c, TSS_ESTATE, "context poisoned by an earlier HIP error");
  if (!c->kv) return fail(c, TSS_ESTATE, "no KV pool bound (tss_kv_alloc)");
  const int np = c->kvl.n_pages;
  if ((int)c->pt_host.size() != np) return fail(c, TSS_ESTATE, "host page table has the wrong length");
  std::vector<uint8_t> seen(np, 0);
  for (int i = 0; i < np; ++i) {
    const int p = c->pt_host[i];
    if (p < 0 || p >= np) return fail(c, TSS_ESTATE, "page table entry " + std::to_string(i) + " outside the pool");
    if (seen[p]++) return fail(c, TSS_ESTATE, "page " + std::to_string(p) + " owned twice");
  }
  std::vector<int32_t> dev(np);
  HIPCHK(hipStreamSynchronize(c->stream), "sync");
  HIPCHK(hipMemcpy(dev.data(), c->kv + c->kvl.page_table, (size_t)np * 4, hipMemcpyDeviceToHost), "page table copy");
  for (int i = 0; i < np; ++i)
    if (dev[i] != c->pt_host[i])
      return fail(c, TSS_ESTATE, "device page table differs from the host copy at entry " + std::to_string(i));
  for (int s = 0; s < c->n_seqs; ++s) {
    if (c->n_kv[s] < 0 || c->n_kv[s] > c->max_tokens)
      return fail(c, TSS_ESTATE, "sequence " + std::to_string(s) + " length outside its capacity");
    for (int l = 0; l < c->cfg.n_layers; ++l)
      if (c->kv_len[s][l] < 0 || c->kv_len[s][l] > c->n_kv[s])
        return fail(c, TSS_ESTATE, "sequence " + std::to_string(s) + " holds K/V past its length");
  }
  return TSS_OK;
}

int tss_get_greedy(tss_ctx* c, int32_t* host_dst, int32_t n_nodes) {
  if (!c || !host_dst) return TSS_EINVAL;
  if (c->poisoned) return fail(c, TSS_ESTATE, "context poisoned by an earlier HIP error");
  if (n_nodes < 1 || n_nodes > c->last_M) return fail(c, TSS_EINVAL, "n_nodes exceeds the last verify's nodes");
  HIPCHK(hipStreamSynchronize(c->stream), "sync");
  HIPCHK(hipMemcpy(host_dst, c->out_ws + c->out_wsl.greedy, (size_t)n_nodes * 4, hipMemcpyDeviceToHost),
         "greedy copy");
  return TSS_OK;
}

}  // extern "C"

// Internal interface of tss_verify_static (tss_static.hip, which holds the
// static scratch).
namespace tss {

int static_prepare(tss_ctx* c, int32_t seq, int* device) {
  const int r = check_ready(c, seq);
  if (r) return r;
  const size_t need = tss_static_workspace_bytes(&c->cfg);
  if (need > (size_t)TSS_STATIC_SCRATCH_BYTES)
    return fail(c, TSS_ENOSPACE,
                "this model's single-sequence workspace (" + std::to_string(need) +
                    " bytes) exceeds the static scratch of " + std::to_string((size_t)TSS_STATIC_SCRATCH_BYTES) +
                    " bytes; use tss_verify with the context's workspace");
  *device = c->device;
  return TSS_OK;
}

int static_hip_fail(tss_ctx* c, hipError_t e, const char* where) { return hip_fail(c, e, where); }

int verify_in_workspace(tss_ctx* c, uint8_t* base, int32_t seq, const int32_t* tokens, const int32_t* parent,
                        int32_t n_nodes, const uint8_t* mask, uint32_t flags, int32_t* accept_len,
                        int32_t* next_token) {
  tss_model_cfg one = c->cfg;
  one.max_batch = 1;
  // the step runs on `base` in the single-sequence layout, with direct
  // launches (a captured step would keep the addresses); the context's own
  // workspace is restored afterwards
  c->ws = base;
  c->wsl = ws_layout(&one);
  c->Mp = round16(row_cap(&one));
  c->direct_only = true;
  const int32_t offs[2] = {0, n_nodes};
  const int r = verify_batch(c, 1, &seq, offs, tokens, parent, mask, flags, accept_len, next_token);
  c->ws = c->ws_own;
  c->wsl = c->wsl_own;
  c->Mp = c->Mp_own;
  c->direct_only = false;
  return r;
}

}  // namespace tss
