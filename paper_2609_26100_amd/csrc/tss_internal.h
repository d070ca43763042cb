// Internal definitions shared by the host runtime and the gfx950 kernels.
//
// Device data layout (all buffers owned by the caller):
//
//   projection inputs (the activation planes of h * gain, attention output,
//   SwiGLU output) are stored tile by tile in MFMA A-operand order
//   (act_index below), Mp rows (a multiple of 16) x K columns per plane.
//
//   packed weights  embed [V][d] (T, row-major, gathered by token id);
//                   per layer: attn_norm [d] f32, W_qkv packed, W_o packed,
//                   mlp_norm [d] f32, W_gateup packed, W_down packed;
//                   final_norm [d] f32; lm_head packed.
//                   A packed matrix W [N][K] is cut into 16-row x KC-column
//                   tiles of exactly 1 KiB (KC = 32 for bf16, 16 for f32),
//                   each stored in MFMA lane order: lane l's 16 bytes are row
//                   (l % 16), columns (l / 16) * KC/4 .. + KC/4 of the tile.
//                   NT adjacent row tiles form a strip; strips are stored one
//                   after the other and, inside a strip, tiles interleave by
//                   K chunk (chunk c of tile t sits at index c * NT + t), so a
//                   wave streaming one strip reads NT KiB contiguous per chunk.
//   workspace       step parameters, residual h [Mp][d] f32, GEMM input
//                   activations, q, attention partials, logits, argmax
//                   partials, greedy tokens, result (offsets in WsLayout).
//   KV pool         page tables, the rotary cos/sin table, then pages.  One
//                   page holds 16 tokens; for (layer, page, head) a K block
//                   [16][hd] (token-major) and a V block [4][hd][4] (token
//                   t at [t / 4][dim][t % 4]), each 16 * hd elements of KV.
//
// Precision modes (T = the packed weights' type):
//   bf16  the caller's bf16 weights are stored as fp16 (T = _Float16; every
//         bf16 value of magnitude 2^-17 .. 65504 converts exactly, smaller
//         ones to the nearest fp16 subnormal, larger ones are refused), and
//         GEMM input activations are one fp16 plane, so the projections are
//         fp16 MFMAs (the paper's precision).  KV cache, q and the attention
//         probabilities are fp16.  Accumulation, residual stream, norms,
//         softmax and logits are fp32.
//   f32   everything fp32 (one activation plane, fp32 KV).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stddef.h>
#include <stdint.h>

struct tss_ctx;

namespace tss {

constexpr int kPage = 16;          // tokens per KV page
constexpr int kMaxNodes = 64;      // nodes of one sequence in one step (u64 ancestor masks)
constexpr int kMaxBatch = 8;       // KV sequences of one step
constexpr int kMaxSegs = 32;       // segments (node sets with their own skip mask) of one step
constexpr int kMaxRows = 128;      // rows (nodes of every segment) of one step
constexpr int kMaxLayers = 256;
constexpr int kTileBytes = 1024;   // one packed 16 x KC weight tile
constexpr int kAttnMaxGroups = 16; // workgroups per (head, sequence) in attention
constexpr int kAttnMaxTiles = 4;   // 16-row tiles of one attention item (64 rows)
constexpr int kAttnMaxItems = 16;  // attention items (row ranges of one KV sequence) of one launch
// attention workgroups one launch of a single sequence aims for: one per CU
// (with cross-workgroup merges through agent-scope accesses, 256 beats the
// 208 that was best while each merge needed device-scope fences: 7B chain
// step 3051 -> 3038 us, 60-node tree 5256 -> 5248 us)
#ifndef TSS_ATTN_TARGET_WGS
#define TSS_ATTN_TARGET_WGS 256
#endif
constexpr int kAttnTargetWGs = TSS_ATTN_TARGET_WGS;
constexpr int kArgPages = 256;     // page ids passed in kernel arguments (one sequence, up to 4096 tokens)
// attention over several KV sequences (a batch): an item takes one workgroup
// per kAttnPagesPerWG pages of its sequence (8 per wave), so a long context
// is walked by several workgroups instead of bounding the launch; all the
// launch's partial-state slots stay within kAttnBatchSlots
constexpr int kAttnPagesPerWG = 64;
// most K splits of one projection launch (the residual projections with
// more than one row tile, see gemm_ksplit)
constexpr int kMaxKSplit = 4;
constexpr int kAttnBatchSlots = 2048;

template <typename T> struct Mode;
template <> struct Mode<_Float16> {
  using KV = _Float16;
  static constexpr int planes = 1;
};
template <> struct Mode<float> {
  using KV = float;
  static constexpr int planes = 1;
};

// Index of element (row, k) of a projection input with K columns (K a
// multiple of the tile width KC = 64 / sizeof(T)), in MFMA A-operand tile
// order: the 16 x KC tile (row / 16, k / KC) is one contiguous KiB whose lane
// l = (k % KC) / (KC / 4) * 16 + row % 16 holds KC / 4 consecutive k, so a
// wave reads a whole tile with one 16-byte load per lane.
template <typename T>
__device__ __forceinline__ size_t act_index(int row, int k, int K) {
  constexpr int KC = 64 / (int)sizeof(T), KL = KC / 4;
  const int nkc = K / KC;
  return (((size_t)(row >> 4) * nkc + k / KC) * 64 + (k % KC) / KL * 16 + (row & 15)) * KL + (k % KL);
}

// Stores an fp32 activation in the mode's plane format.
template <typename T>
__device__ __forceinline__ void store_act(void* base, size_t plane, size_t idx, float v) {
  if constexpr (Mode<T>::planes == 2) {
    const T hi = (T)v;
    ((T*)base)[idx] = hi;
    ((T*)base)[plane + idx] = (T)(v - (float)hi);
  } else {
    ((T*)base)[idx] = (T)v;
  }
}

// Stores activations k .. k+3 of one row (k a multiple of 4), which act_index
// places next to each other in each plane: one 8-byte (16-bit planes) or
// 16-byte (f32) store per plane instead of one per element.
// idx = act_index(row, k).
template <typename T>
__device__ __forceinline__ void store_act4(void* base, size_t plane, size_t idx, float4 v) {
  if constexpr (Mode<T>::planes == 2) {
    const T h0 = (T)v.x, h1 = (T)v.y, h2 = (T)v.z, h3 = (T)v.w;
    const T l0 = (T)(v.x - (float)h0), l1 = (T)(v.y - (float)h1), l2 = (T)(v.z - (float)h2), l3 = (T)(v.w - (float)h3);
    typedef T t4 __attribute__((ext_vector_type(4)));
    *(t4*)((T*)base + idx) = t4{h0, h1, h2, h3};
    *(t4*)((T*)base + plane + idx) = t4{l0, l1, l2, l3};
  } else if constexpr (sizeof(T) == 4) {
    *(float4*)((T*)base + idx) = v;
  } else {
    typedef T t4 __attribute__((ext_vector_type(4)));
    *(t4*)((T*)base + idx) = t4{(T)v.x, (T)v.y, (T)v.z, (T)v.w};
  }
}

// Per-step data that changes from step to step (tokens, tree, context
// lengths).  Rows are grouped into segments: the nodes of one draft tree
// verified under one skip mask, numbered locally from 0 (its root), segment
// after segment.  A segment belongs to one KV sequence; several segments of
// one sequence (one context verified under several masks) sit next to each
// other and take consecutive draft slots after the context: node j of
// segment s has slot seq_nkv[s] + seg_slot0[s] + j.  In a plain batch every
// segment is its own sequence and seg_slot0 is 0.
struct StepParams {
  int32_t M;                       // rows
  int32_t n_seqs;                  // segments
  int32_t seq_row0[kMaxSegs + 1];  // first row of each segment; seq_row0[n_seqs] = M
  int32_t seq_nkv[kMaxSegs];       // committed context length of each segment's sequence
  int32_t tok[kMaxRows];
  uint64_t anc[kMaxRows];          // bit j: local node j is this node or one of its ancestors
  int8_t parent[kMaxRows];         // local parent (-1 for the root)
  uint8_t depth[kMaxRows];
  uint8_t row_seq[kMaxRows];       // segment (0 .. n_seqs-1) of the row
  uint8_t seg_slot0[kMaxSegs];     // first draft slot of each segment, after its sequence's context
  uint8_t row_slot0[kMaxRows];     // seg_slot0 of the row's segment
};

// Position of a row: its sequence's committed length plus its depth.
__device__ __forceinline__ int row_pos(const StepParams* sp, int row) {
  return sp->seq_nkv[sp->row_seq[row]] + sp->depth[row];
}

struct Result {
  int32_t accept_len;
  int32_t next_token;
  int32_t best;
  int32_t path_len;                // accept_len + 1
  int32_t path[kMaxNodes];         // local node ids root -> best
};

enum Epi { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3 };

struct GemmArgs {
  const uint8_t* w;        // packed weights of this matrix
  const void* x;           // A operand [Mp][K] of T in tile order (act_index), planes x_plane elements apart
  size_t x_plane;
  int M, K, N;             // N = packed output columns
  int nkc;                 // K / KC
  // RMSNorm of the A rows: x holds T(h * gain); the row scale
  // rsqrt(sum(h^2) / norm_dim + eps) is applied to the products here.
  const float* ss_in;      // [M][ss_stride] partial sums of h^2, ss_nparts used (null: no norm)
  int ss_nparts;
  int ss_stride;           // row stride of ss_in / ss_out (parts)
  int norm_dim;
  float eps;
  int Mp;                  // row stride of the partial-sum arrays
  // K split (> 1): workgroup blockIdx.x takes strip blockIdx.x / ksplit over
  // its share of K; the ksplit partial products of a strip meet in kpart
  // (agent-scope accesses) and the last workgroup to arrive finishes the strip
  int ksplit;
  // gate/up in blocks of two widths (gemm_wide_wgs > 0): workgroups
  // [0, wide_wgs) take NT / 2 pairs, the rest NT / 2 - 1
  int wide_wgs;
  float* kpart;            // [strips * ksplit][Mp][16 * NT] partial products
  int* kcount;             // [strips] arrivals, zero between launches
  const StepParams* sp;
  // rows whose segment runs this block (bit r of row_on[r / 64]); the QKV
  // and residual epilogues write nothing for the other rows
  uint64_t row_on[kMaxRows / 64];
  int n_seqs;              // segments
  // EPI_QKV
  float* q;                // [Mp][d]
  uint8_t* kv_pages;       // first page of the pool
  const int32_t* page_table;  // the pool's page table; segment s's sequence's pages start at pt_off[s]
  int32_t pt_off[kMaxSegs];
  int32_t n_arg_pages;     // with one KV sequence in the step: valid entries of pages[] (else 0)
  int32_t pages[kArgPages];  // physical ids of that sequence's first pages
  const float2* rope;      // [max_pos][hd/2] (cos, sin)
  int layer, n_pages_pool, n_heads, head_dim, d;
  // EPI_RESID
  float* h;                // [Mp][N] residual, updated in place
  void* xn;                // [Mp][N] activation planes of h_new * g_next
  size_t xn_plane;
  const float* g_next[kMaxSegs];   // gain of each segment's next RMSNorm
  float* ss_out;           // [M][ss_stride] partial sums of h_new^2, one per strip
  // EPI_SWIGLU
  void* act;               // [Mp][N/2] activation planes of silu(gate) * up
  size_t act_plane;
  // EPI_LOGITS
  float* logits;           // [Mp][N]
  float* am_val;           // [M][am_stride] per-strip (max, argmax)
  int32_t* am_idx;
  int am_stride;
};

// An attention item is a range of at most 64 consecutive rows of one KV
// sequence (grid.y walks the items): its workgroups read the sequence's pages
// once for all of its rows, whatever segments they belong to.
struct AttnArgs {
  const float* q;          // [Mp][d] row-major
  const uint8_t* kv_pages;
  const int32_t* page_table;
  const StepParams* sp;
  void* o;                 // activation planes of the attention output (act_index order)
  size_t o_plane;
  // partial states, slot ((head * n_items + y) * groups + g), kAttnMaxTiles tiles each
  float* part_o;           // [slots][kAttnMaxTiles][16][hd] unnormalised partial outputs
  float* part_ml;          // [slots][kAttnMaxTiles][16][2] (max in log2 units, sum)
  int* counters;           // [H * kAttnMaxItems] arrivals, zero between launches
  // report of the launch's split: per item the workgroups G its pages were
  // divided among and its rows, then the item count ([2 * kAttnMaxItems + 1])
  int32_t* split_out;
  int groups;              // most workgroups per (head, item)
  int pages_per_wg;        // > 0: an item takes ceil(pages / pages_per_wg) workgroups (at most groups)
  int defer_merge;         // partial states merged by a second launch (launches with items of 2+ row tiles)
  int layer, n_pages_pool, n_heads, d;
  float scale_log2;        // log2(e) / sqrt(hd)
  // per item, 32-bit so that the kernel reads them with scalar loads
  int32_t item_row0[kAttnMaxItems];   // first row of the item
  int32_t item_rows[kAttnMaxItems];   // rows (1 .. 64)
  int32_t item_seg[kAttnMaxItems];    // segment of the first row (context length, page table)
  int32_t item_slots[kAttnMaxItems];  // draft slots after the context that its rows may see
  int32_t pt_off[kMaxSegs];
  int32_t n_arg_pages;     // with one KV sequence in the step: valid entries of pages[] (else 0)
  int32_t pages[kArgPages];  // physical ids of that sequence's first pages
};

struct EmbedArgs {
  const void* embed;       // [V][d] T
  // when set, row m starts from a saved residual instead of its token's
  // embedding: src_h[j][d] fp32 with j = m's local node (a step that resumes
  // after blocks every segment shares with the dense verifier)
  const float* src_h;
  StepParams sp;           // this step's parameters (by value) ...
  StepParams* sp_dev;      // ... copied here for the later kernels of the step
  const float* gain[kMaxSegs];   // per segment: gain of the first RMSNorm its rows meet
  float* h;                // [Mp][d]
  void* xn;                // [Mp][d] activation planes
  size_t xn_plane;
  float* ss_out;           // [M][ss_stride]: sums of h^2 over 16-column parts
  int ss_stride;
  int d, M;
  int32_t* attn_split;     // the attention split report (AttnArgs::split_out): its item count is cleared
  int32_t* counters;       // arrival counters of the step's merges (attention, K split), cleared here
  int n_counters;
};

struct AcceptArgs {
  const float* am_val;     // [M][am_stride]
  const int32_t* am_idx;
  int nparts, M, am_stride;
  const StepParams* sp;
  int32_t* greedy;         // [Mp] (agent-scope stores: the last row's workgroup reads them all)
  int* count;              // rows finished, zero between launches
  Result* result;          // [n_seqs] device copy, one per segment (read by the compaction kernel)
  Result* result_host;     // [n_seqs] host-mapped pinned copy (read by the host after the step)
};

struct CompactArgs {
  uint8_t* kv_pages;
  const int32_t* page_table;
  const StepParams* sp;
  const Result* result;    // [n_seqs]
  int n_layers, n_pages_pool, n_heads, head_dim;
  // grid.z walks the sequences listed here (those whose accepted tree path
  // needs moving); lay_on[i] has bit l set for each layer sequence seq[i] ran
  int32_t seq[kMaxBatch];
  int32_t pt_off[kMaxBatch];
  uint64_t lay_on[kMaxBatch][kMaxLayers / 64];
};

// Events bound to the next launch's own dispatch (profiling).  When `start` is
// set, TSS_LAUNCH issues the kernel through hipExtLaunchKernel, which stamps
// the two events with the start and end of the kernel's execution, the same
// dispatch timestamps a kernel-trace profiler reports; otherwise it is a plain
// launch.  Set only around direct (not captured) launches.
struct LaunchTiming {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchTiming& launch_timing();

#define TSS_LAUNCH(kernel, grid, block, lds, stream, ...)                                          \
  do {                                                                                             \
    const ::tss::LaunchTiming& lt_ = ::tss::launch_timing();                                       \
    if (lt_.start)                                                                                 \
      hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)(lds), stream, lt_.start, lt_.stop, 0u, \
                            __VA_ARGS__);                                                          \
    else                                                                                           \
      hipLaunchKernelGGL(kernel, grid, block, lds, stream, __VA_ARGS__);                           \
  } while (0)

// Launchers (defined in the .hip files).  T is selected by `bf16`.
hipError_t launch_gemm(bool bf16, int epi, int mt, int nt, const GemmArgs& a, hipStream_t s);
hipError_t launch_attn(bool bf16, int head_dim, int max_tiles, int n_items, const AttnArgs& a, hipStream_t s);
hipError_t launch_embed(bool bf16, const EmbedArgs& a, hipStream_t s);
hipError_t launch_accept(const AcceptArgs& a, hipStream_t s);
hipError_t launch_compact(bool bf16, int n_seqs, const CompactArgs& a, hipStream_t s);
const void* embed_kernel(bool bf16);  // kernel symbol, for updating a captured launch
hipError_t init_kernel_attributes();  // attention
hipError_t init_gemm_attributes();
hipError_t launch_rope_table(float2* tab, int max_pos, int head_dim, float base, hipStream_t s);

// Host runtime pieces of tss_verify_static (tss_static.hip holds the static
// scratch): the checks before any device work (sequence state, the model's
// single-sequence workspace against the scratch size; the context's device),
// the error of a failed HIP call, and a single-sequence verify whose step
// workspace is `base` (direct launches; the context's own workspace is
// restored afterwards).
int static_prepare(tss_ctx* c, int32_t seq, int* device);
int static_hip_fail(tss_ctx* c, hipError_t e, const char* where);
int verify_in_workspace(tss_ctx* c, uint8_t* base, int32_t seq, const int32_t* tokens, const int32_t* parent,
                        int32_t n_nodes, const uint8_t* mask, uint32_t flags, int32_t* accept_len,
                        int32_t* next_token);

// Workgroups of one projection round on this GPU (one per CU).
constexpr int kGemmRound = 256;

// Gate/up in one round of 256 workgroups of two block widths: with 2-4 row
// tiles where the pairs (N / 32) lie between two and three per workgroup,
// three pairs (six tiles) for the first `pairs - 512` workgroups and two for
// the rest (7B: 176 x 3 + 80 x 2 pairs instead of 172 x 4, which left CUs
// idle); with 5 row tiles where they lie between three and four, four and
// three pairs (13B: 96 x 4 + 160 x 3 instead of 432 x 2 in two rounds).
// Returns that count of wider workgroups, or 0.
inline int gemm_wide_pairs(int epi, int mt, int N) {
  if (epi != EPI_SWIGLU || N % 32) return 0;
  const int pairs = N / 32;
  if (mt >= 2 && mt <= 4 && pairs > 2 * kGemmRound && pairs <= 3 * kGemmRound) return 3;
  if (mt == 5 && pairs > 3 * kGemmRound && pairs <= 4 * kGemmRound) return 4;
  return 0;
}
inline int gemm_wide_wgs(int epi, int mt, int N) {
  const int w = gemm_wide_pairs(epi, mt, N);
  return w ? N / 32 - (w - 1) * kGemmRound : 0;
}

// 16-column tiles per workgroup of a projection launch.  A workgroup streams
// its tiles over all of K, so every workgroup reads all of the step's
// activation tiles: a wider block makes each activation tile serve more
// weight tiles, but leaves fewer workgroups.  Measured on the 7B, 13B and
// 33B shapes (6 to 72 rows): the best width is the narrowest that fits the
// matrix in one round of at most 256 workgroups (with more than one row tile
// a workgroup fills a CU), except that with one row tile gate/up keeps one
// gate/up pair, lm_head one tile, and Q/K/V takes 4 tiles only if that fits
// 256 workgroups (else 2), and Q/K/V takes 3 tiles when that gives more than
// 192 and at most 256 workgroups (7B: 256 instead of 192; the 7B k=5 step
// 3133 -> 3096 us, the 60-node tree 5903 -> 5792 us); with 2-4 row tiles
// gate/up takes 8 tiles when they fit 256 workgroups (the 60-node tree
// 5851 -> 5531 us), or blocks of two widths that fill the round exactly
// (gemm_wide_pairs), and lm_head 8 tiles where 4 would need two rounds.
// The residual projections with 2-8 row tiles take four- (two-) tile blocks
// over a share of K instead (gemm_ksplit; the partial tiles meet through agent-scope
// accesses, with no device-scope fence).
inline int gemm_tiles(int epi, int mt, int N) {
  if (gemm_wide_pairs(epi, mt, N) > 0) return 2 * gemm_wide_pairs(epi, mt, N);  // blocks of two widths
  // residual projections with 2-7 row tiles: four-tile blocks over a share of
  // K (gemm_ksplit), so each workgroup re-reads a quarter of the activation
  // tiles that a one-tile block over all of K would
  if (epi == EPI_RESID && mt >= 2 && mt <= 7 && N % 64 == 0) return 4;
  // eight row tiles: two-tile blocks (four would spill), split where that
  // fills the round (7B: 128 strips x 2; 7B 64-mask sweep 16.05 -> 14.97 ms)
  if (epi == EPI_RESID && mt == 8 && N % 32 == 0 && N / 32 <= 256) return 2;
  // gate/up with 2-4 row tiles: eight-tile blocks (four pairs) when they fit
  // one round (7B: 172 workgroups instead of 344 in 1.34 rounds; more row
  // tiles would spill)
  if (epi == EPI_SWIGLU && mt >= 2 && mt <= 4 && N % 128 == 0 && N / 128 <= 256) return 8;
  // the same for the wider matrices (33B): ten-tile gate/up blocks with 2-3
  // row tiles, six-tile Q/K/V blocks with 2-4, where four-tile ones would take
  // more than one round (33B: 224 instead of 560 and 208 instead of 312
  // workgroups; the 33B single-mask step 18.1 -> 14.9 ms)
  if (epi == EPI_SWIGLU && mt >= 2 && mt <= 3 && N % 160 == 0 && N / 160 <= 256 && N / 160 > 192) return 10;
  if (epi == EPI_QKV && mt >= 2 && mt <= 4 && N % 96 == 0 && N / 96 <= 256 && N / 96 > 192 && N / 64 > 256) return 6;
  if (epi == EPI_SWIGLU) return (mt == 1 || N % 64) ? 2 : 4;
  if (mt == 1 && epi == EPI_LOGITS) return 1;
  // lm_head with 2-4 row tiles: eight-tile blocks in one round where four-tile
  // ones need two (32000-token vocabulary: 250 instead of 500 workgroups;
  // with 5 row tiles they would spill)
  if (epi == EPI_LOGITS && mt >= 2 && mt <= 4 && N % 128 == 0 && N / 128 <= 256 && N / 64 > 256) return 8;
  // one row tile: one-tile Q/K/V blocks three to a CU where they fill one
  // such round (7B: 768 workgroups; the 7B k=5 step -20 us against 256
  // three-tile blocks, one per CU)
  if (epi == EPI_QKV && mt == 1 && N % 16 == 0 && N / 16 <= 768 && N / 16 > 512) return 1;
  // three-tile Q/K/V blocks where they fill one round better than four-tile
  // ones can (more than 192 and at most 256 workgroups: the 7B shape's 256)
  if (epi == EPI_QKV && N % 48 == 0 && N / 48 <= 256 && N / 48 > 192) return 3;
  if (mt == 1 && epi == EPI_QKV) return (N % 64 == 0 && N / 64 <= 256) ? 4 : (N % 32 == 0 ? 2 : 1);
  for (int nt = 1; nt <= 4; nt *= 2)
    if (N % (16 * nt) == 0 && N / (16 * nt) <= 256) return nt;
  return N % 64 == 0 ? 4 : (N % 32 == 0 ? 2 : 1);
}

// K splits of a projection launch: the residual projections with 2-7 row
// tiles split K so that their four-tile blocks still fill about one round of
// 256 workgroups (7B: 64 strips x 4, 13B: 80 x 3, 33B: 104 x 2), and with 8
// row tiles their two-tile blocks (7B: 128 x 2), each split keeping at least
// one chunk per wave.  nkc = K chunks of the matrix.
inline int gemm_ksplit(int epi, int mt, int N, int nkc) {
  const bool four = epi == EPI_RESID && mt >= 2 && mt <= 7 && N % 64 == 0;
  const bool two = epi == EPI_RESID && mt == 8 && N % 32 == 0 && N / 32 <= 256;
  if (!four && !two) return 1;
  int ks = 256 / (N / (four ? 64 : 32));
  ks = ks < 1 ? 1 : (ks > kMaxKSplit ? kMaxKSplit : ks);
  while (ks > 1 && nkc / ks < 8) --ks;
  return ks;
}

}  // namespace tss
