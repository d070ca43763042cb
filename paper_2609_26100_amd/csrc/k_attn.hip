// Tree-masked attention of the verify step over the paged KV cache (gfx950).
//
// For every head and node i of a segment: softmax(q_i K^T / sqrt(hd)) V over
// its sequence's cached context [0, n_kv) plus the segment's draft nodes
// visible to i (i itself and its ancestors; the QKV kernel appended their K/V
// at the segment's draft slots n_kv + slot0 + j).  This is the attention half
// of an active block; bypassed blocks never reach this kernel (Domain-Aware
// Skip Controller, block rule).
//
// grid = (head, item, workgroup of that item).  An item is up to 64
// consecutive rows of one KV sequence, possibly from several segments (one
// context verified under several skip masks).  An item's G workgroups of 8
// waves split the sequence's pages (wave w of workgroup g walks pages
// 8 g + w, 8 (g + G) + w, ..., loading the next page while it computes the
// current one), and each wave applies every page to all of the item's row
// tiles (up to 4 x 16 rows), so each K/V page is read from HBM once per head
// however many nodes and masks the item carries.  (Serving the tiles from
// different waves instead measured slower: more page loads per tile.)
//   * The K page block [16 tokens][hd] is read with one contiguous 64-byte run
//     per lane (the whole 4 KiB block per wave), and S = K Q^T comes out of
//     MFMA with tokens on the rows and nodes on the columns.
//   * The S accumulator layout (lane: node column, 4 token rows) is exactly
//     the A-operand layout of the P V product, so probabilities never leave
//     registers.  The V block is stored [4][hd][4] so each lane's B operand for
//     all hd/16 output tiles is again one contiguous 64-byte run.
//   * Online softmax in the exp2 domain, fp32; masked keys get -inf.
//   * Operands: fp16 K/V pages, q and probabilities with fp32 accumulation
//     (v_mfma_f32_16x16x32_f16 for S, v_mfma_f32_16x16x16_f16 for P V) in the
//     bf16 mode; fp32 throughout (v_mfma_f32_16x16x4_f32) in the f32 mode.
// The 8 waves' softmax states meet in LDS (fixed order), tile after tile.
// With G = 1 the workgroup writes the normalised rows itself.  With G > 1,
// in launches of single-tile items, each workgroup writes its partial states
// with agent-scope stores, waits for them to land, and bumps a per-(head,
// sequence) counter; the last to arrive reads them with agent-scope loads and
// merges the G partials in workgroup order and resets the counter (no second
// kernel: a kernel boundary costs about as much as this hand-over).  Items of
// several row tiles have too many partial states for one workgroup to read
// quickly (256 KiB at four tiles and eight workgroups: 8.4 us), so their
// launches leave the partial states to k_attn_merge, a second launch in which
// each workgroup merges 8 rows of one (head, item).  Either way the order of
// summation is fixed: results are bit-reproducible.
//
// An item's G (at most `groups`, at least one page per wave, at most
// pages / (4 T), and in a batch of sequences one per `pages_per_wg` pages) is
// derived on the device from its context length, so launch arguments do not
// depend on context lengths; workgroups beyond an item's G exit at once.
#include "tss_internal.h"

namespace tss {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ unsigned pack_f16x2(float lo, float hi) {
  const _Float16 a = (_Float16)lo, b = (_Float16)hi;
  return (unsigned)__builtin_bit_cast(unsigned short, a) | ((unsigned)__builtin_bit_cast(unsigned short, b) << 16);
}

// Reductions over the four lanes l, l^16, l^32, l^48 of a node column with
// gfx950's row-swap permutes (VALU, no trip through the LDS pipeline): given
// one value twice, v_permlane16_swap leaves a lane its own value and that of
// the lane 16 away, v_permlane32_swap its own and that of the lane 32 away.
// Max and sum are commutative, so every lane gets the same bits as with
// pairwise exchanges.
__device__ __forceinline__ float max_col4(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  const auto h = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(h[0]), __uint_as_float(h[1]));
}
__device__ __forceinline__ float sum_col4(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  const auto h = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(h[0]) + __uint_as_float(h[1]);
}

// Partial states travel between workgroups (possibly on different XCDs, whose
// L2 caches are not coherent with each other) through agent-scope accesses:
// the stores write through to the level every XCD sees and the loads read
// from it (scope bit sc1), so publishing them needs no L2 write-back or
// invalidation.  The partial outputs go through a buffer resource (one
// 16-byte access per four floats); offsets are in bytes.
constexpr int kScopeAgent = 16;  // cache-policy operand of buffer accesses: sc1
__device__ __forceinline__ void store_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_agent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_agent4(__amdgpu_buffer_rsrc_t r, int off, float4 v) {
  typedef float f4v __attribute__((ext_vector_type(4)));
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(f4v, v), r, off, 0, kScopeAgent);
}
__device__ __forceinline__ float4 load_agent4(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kScopeAgent));
}

#ifndef TSS_ATTN_WAVES
#define TSS_ATTN_WAVES 8
#endif
#ifndef TSS_ATTN_PART_DIV
#define TSS_ATTN_PART_DIV 4
#endif
constexpr int kAttnWaves = TSS_ATTN_WAVES;

// Workgroups an item's n_pages pages are divided among: at most `groups`, at
// least a page per wave, few enough that the partial states (T tiles each)
// stay well below the pages, and in a batch of sequences one per
// pages_per_wg pages.  The attention and merge launches derive it alike.
__device__ __forceinline__ int attn_item_groups(const AttnArgs& a, int n_pages, int T) {
  const int cap = a.pages_per_wg > 0 ? min(a.groups, (n_pages + a.pages_per_wg - 1) / a.pages_per_wg) : a.groups;
  return max(1, min(cap, min((n_pages + kAttnWaves - 1) / kAttnWaves, n_pages / (TSS_ATTN_PART_DIV * T))));
}

// Dynamic LDS: q tiles [TMAX][64][NQ] uint4 | m, l [W][16] | O [W][64][OS].
// The paired walk over an fp16 KV cache keeps the same areas in static
// arrays instead: during the walk the O area holds each wave's LDS page
// slot, written by global -> LDS loads, and with distinct static arrays the
// compiler can tell those writes from the walk's other LDS accesses (so
// reading q does not wait for page loads in flight).
template <typename TK, int HD, int TMAX, bool PAIR>
constexpr size_t attn_lds() {
  constexpr int NQ = HD / 4 * (int)sizeof(TK) / 16;
  constexpr int OS = HD / 16 * 4 + 1;
  return PAIR && sizeof(TK) == 2 ? 0 : (size_t)(TMAX * 64 * NQ * 4 + kAttnWaves * 16 * 2 + kAttnWaves * 64 * OS) * 4;
}
typedef __attribute__((address_space(1))) const void global_cvoid;
typedef __attribute__((address_space(3))) void lds_void;

// TK = KV element type (_Float16 or float); TW = weight type of the mode
// (selects the activation plane format of the output); TMAX = most node
// tiles of an item in this launch; PAIR = the paired page walk (launches
// over one KV sequence; with several sequences the walk with one page ahead
// in registers measured faster: 13B batch of 8 9.71 against 10.04 ms).
template <typename TK, typename TW, int HD, int TMAX, bool PAIR>
__global__ __launch_bounds__(kAttnWaves * 64) void k_attn(AttnArgs a) {
  constexpr int DL = HD / 4;                         // dims per lane group in Q K^T
  constexpr int NQ = DL * (int)sizeof(TK) / 16;      // 16-byte K/Q chunks per lane
  constexpr int NO = HD / 16;                        // output tiles of P V
  constexpr int NV = NO * 4 * (int)sizeof(TK) / 16;  // 16-byte V chunks per lane
  constexpr int W = kAttnWaves;
  constexpr int OS = NO * 4 + 1;

  const int head = blockIdx.x, y = blockIdx.y, g = blockIdx.z;
  // The wave index is uniform, so page ids and page addresses come from
  // scalar loads, whose waits never hold back page loads in flight.
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63, r16 = lane & 15,
            grp = lane >> 4;
  const int arg_pages = a.n_arg_pages;
  const int32_t* pt = a.page_table;  // this item's row of the page table, set below

  // With the paired walk all of the kernel's LDS is static (see attn_lds):
  // q tiles, m and l in s_qml, the merge area [W][64][OS] in s_o, which
  // holds the waves' page slots during the walk
  constexpr bool kLdsWalk = PAIR && sizeof(TK) == 2;
  __shared__ __align__(16) float s_o[kLdsWalk ? W * 64 * OS : 4];
  __shared__ __align__(16) float s_qml[kLdsWalk ? TMAX * 64 * NQ * 4 + W * 16 * 2 : 4];

  const size_t blk_elems = 16 * (size_t)HD;
  auto load_phys = [&](int phys, uint4 (&kreg)[NQ], uint4 (&vreg)[NV]) {
    const TK* kb = (const TK*)a.kv_pages + (((size_t)a.layer * a.n_pages_pool + phys) * 2 * a.n_heads + head) * blk_elems;
    const TK* vb = kb + (size_t)a.n_heads * blk_elems;
    const uint4* kp = (const uint4*)(kb + r16 * HD + grp * DL);
    const uint4* vp = (const uint4*)(vb + grp * HD * 4 + r16 * NO * 4);
#pragma unroll
    for (int c = 0; c < NQ; ++c) kreg[c] = kp[c];
#pragma unroll
    for (int c = 0; c < NV; ++c) vreg[c] = vp[c];
  };
  // Page p of the item's sequence, the wave's it-th page.  p is uniform: the
  // argument list is read with a scalar load; pages past it take their id
  // from `ids` (lane it holds the id of the wave's it-th page, read with one
  // vector load before the walk, so the walk never waits on a page-table
  // read) or, past the wave's 64th page, from the page table.
  int ids = 0;
  auto page_phys = [&](int p, int it) {
    if (p < arg_pages) return a.pages[p];
    if (it < 64) return __builtin_amdgcn_readlane(ids, it);
    return __builtin_amdgcn_readfirstlane(__builtin_nontemporal_load(pt + p));
  };
  auto load_page = [&](int p, int it, uint4 (&kreg)[NQ], uint4 (&vreg)[NV]) {
    load_phys(page_phys(p, it), kreg, vreg);
  };
  // The same page into the wave's LDS slot (global -> LDS, no registers):
  // 16-byte chunk c of lane l lands at pslot[c * 64 + l], K chunks first,
  // where the walk reads it back into the registers load_phys would fill.
  // Every wave's slot lies inside its own row range of the merge area
  // ((NQ + NV) KiB <= 64 * OS floats).
  uint4* const pslot = (uint4*)(s_o + (kLdsWalk ? wave * 64 * OS : 0));
  static_assert(!kLdsWalk || (NQ + NV) * 64 * 16 <= 64 * OS * 4, "page slot inside the wave's merge rows");
  auto dma_page = [&](int p, int it) {
    const int phys = page_phys(p, it);
    const TK* kb = (const TK*)a.kv_pages + (((size_t)a.layer * a.n_pages_pool + phys) * 2 * a.n_heads + head) * blk_elems;
    const TK* vb = kb + (size_t)a.n_heads * blk_elems;
    const uint4* kp = (const uint4*)(kb + r16 * HD + grp * DL);
    const uint4* vp = (const uint4*)(vb + grp * HD * 4 + r16 * NO * 4);
#pragma unroll
    for (int c = 0; c < NQ; ++c)
      __builtin_amdgcn_global_load_lds((global_cvoid*)(kp + c), (lds_void*)(pslot + c * 64), 16, 0, 0);
#pragma unroll
    for (int c = 0; c < NV; ++c)
      __builtin_amdgcn_global_load_lds((global_cvoid*)(vp + c), (lds_void*)(pslot + (NQ + c) * 64), 16, 0, 0);
  };

  // The wave's first page is requested before anything else when its id is
  // an argument: every argument id names a page of the pool, so the load is
  // in bounds even if the page lies past the context (its data is then never
  // used).  Its latency overlaps the reads of the item's parameters, q and
  // the tree masks below.
  uint4 kcur[NQ], vcur[NV];
  int p = g * W + wave;
  const bool early = p < arg_pages;
  if (early) load_phys(a.pages[p], kcur, vcur);

  const int sq = a.item_seg[y];
  const int n_kv = a.sp->seq_nkv[sq];
  const int row0 = a.item_row0[y];
  const int Ms = a.item_rows[y];                     // rows of the item
  const int T = (Ms + 15) >> 4;                      // its row tiles (<= TMAX)
  const int n_pages = (n_kv + a.item_slots[y] + kPage - 1) / kPage;
  const int G = attn_item_groups(a, n_pages, T);
  if (head == 0 && g == 0 && threadIdx.x == 0) {  // the split this launch took (inspection)
    a.split_out[y] = G;
    a.split_out[kAttnMaxItems + y] = Ms;
    if (y == 0) a.split_out[2 * kAttnMaxItems] = (int)gridDim.y;
  }
  if (g >= G) {                                      // uniform over the workgroup
    __builtin_amdgcn_s_waitcnt(0);                   // let the early page load land first
    return;
  }
  pt = a.page_table + a.pt_off[sq];
  const int stride = W * G;
  if (n_pages > arg_pages) {  // uniform: some page of the item lies past the argument list
    const int pp = p + lane * stride;
    if (pp < n_pages && pp >= arg_pages) ids = __builtin_nontemporal_load(pt + pp);
  }

  // B operand of S = K Q^T for tile t: lane (node 16 t + r16, group grp)
  // holds q[node][head*HD + grp*DL + 0..DL).  Waves 0..T-1 build one tile
  // each in LDS (all of a lane's loads issued before the first conversion);
  // every wave re-reads them per page.
  extern __shared__ float smem_dyn[];
  float* const smem = kLdsWalk ? s_qml : smem_dyn;
  uint4* sm_q = (uint4*)smem;  // [TMAX][64][NQ]
  if (wave < T) {
    const int ln = wave * 16 + r16;  // local node
    const float* qrow = a.q + (size_t)(row0 + ln) * a.d + head * HD + grp * DL;
    constexpr int NF = DL / 4;       // float4 loads per lane
    float4 f[NF];
    if (ln < Ms) {
#pragma unroll
      for (int i = 0; i < NF; ++i) f[i] = *(const float4*)(qrow + i * 4);
    } else {
#pragma unroll
      for (int i = 0; i < NF; ++i) f[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int c = 0; c < NQ; ++c) {
      uint4 qv;
      if constexpr (sizeof(TK) == 2) {
        const float4 f0 = f[2 * c], f1 = f[2 * c + 1];
        qv = uint4{pack_f16x2(f0.x, f0.y), pack_f16x2(f0.z, f0.w), pack_f16x2(f1.x, f1.y), pack_f16x2(f1.z, f1.w)};
      } else {
        qv = __builtin_bit_cast(uint4, f[c]);
      }
      sm_q[(wave * 64 + lane) * NQ + c] = qv;
    }
  }
  // draft visibility of row (tile t, r16): slot n_kv + base[t] + j holds its
  // segment's node j, visible when bit j of anc[t] is set
  uint64_t anc[TMAX];
  int base[TMAX];
#pragma unroll
  for (int t = 0; t < TMAX; ++t) {
    const int ln = t * 16 + r16;
    const bool in = t < T && ln < Ms;
    anc[t] = in ? a.sp->anc[row0 + ln] : 0ull;
    base[t] = in ? (int)a.sp->row_slot0[row0 + ln] : 0;
  }

  float m_run[TMAX], l_run[TMAX];
  f32x4 O[TMAX][NO];
#pragma unroll
  for (int t = 0; t < TMAX; ++t) {
    m_run[t] = -1e30f;
    l_run[t] = 0.f;
#pragma unroll
    for (int n = 0; n < NO; ++n) O[t][n] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  if (!early && p < n_pages) load_page(p, 0, kcur, vcur);
  float* sm_alpha = smem + TMAX * 64 * NQ * 4 + wave * 16;  // the wave's slots of the merge's m array
  // Folds page pg (K chunks in kc, V chunks in vc) into every row tile's
  // online-softmax state.
  auto walk_page = [&](int pg, const uint4 (&kc)[NQ], const uint4 (&vc)[NV]) {
#pragma unroll
    for (int t = 0; t < TMAX; ++t) {
      if (t >= T) break;
      f32x4 S = f32x4{0.f, 0.f, 0.f, 0.f};
      asm volatile("" ::: "memory");  // re-read the q tile from LDS each page (keeps it out of registers)
#pragma unroll
      for (int c = 0; c < NQ; ++c) {
        const uint4 qv = sm_q[(t * 64 + lane) * NQ + c];
        if constexpr (sizeof(TK) == 2) {
          S = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, kc[c]),
                                                     __builtin_bit_cast(f16x8, qv), S, 0, 0, 0);
        } else {
          S = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kc[c].x), __uint_as_float(qv.x), S, 0, 0, 0);
          S = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kc[c].y), __uint_as_float(qv.y), S, 0, 0, 0);
          S = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kc[c].z), __uint_as_float(qv.z), S, 0, 0, 0);
          S = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kc[c].w), __uint_as_float(qv.w), S, 0, 0, 0);
        }
      }

      // S[v] = score of token 4*grp+v of this page against local node 16 t + r16.
      // Only pages that reach past the context hold draft slots, whose
      // visibility depends on the node (pg is uniform, so is the branch).
      float s[4];
      float mloc;
      if ((pg + 1) * kPage <= n_kv) {
#pragma unroll
        for (int v = 0; v < 4; ++v) s[v] = S[v] * a.scale_log2;
        mloc = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
      } else {
        mloc = -INFINITY;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int slot = pg * kPage + grp * 4 + v;
          bool vis;
          if (slot < n_kv) {
            vis = true;
          } else {
            const unsigned j = (unsigned)(slot - n_kv - base[t]);
            vis = j < 64u && ((anc[t] >> j) & 1ull);
          }
          s[v] = vis ? S[v] * a.scale_log2 : -INFINITY;
          mloc = fmaxf(mloc, s[v]);
        }
      }
      // exponentials with the bare v_exp_f32 (results below 2^-126 flush to
      // zero, which no probability or weight here needs)
      const float m_new = fmaxf(m_run[t], max_col4(mloc));
      const float alpha = __builtin_amdgcn_exp2f(m_run[t] - m_new);
      float pv[4];
      float lsum = 0.f;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        pv[v] = __builtin_amdgcn_exp2f(s[v] - m_new);
        lsum += pv[v];
      }
      l_run[t] = l_run[t] * alpha + sum_col4(lsum);
      m_run[t] = m_new;

      // O rows are nodes 4*grp+v; their rescale factors (one per node column)
      // pass through this wave's 16 LDS floats: written by the lanes of
      // group 0, read back as one 16-byte load (a wave's LDS accesses complete
      // in order, so no barrier is needed; the merge's m slots are free until
      // the walk ends).
      if (grp == 0) sm_alpha[r16] = alpha;
      __builtin_amdgcn_wave_barrier();
      const float4 av4 = *(const float4*)(sm_alpha + grp * 4);
      __builtin_amdgcn_wave_barrier();
      const float av[4] = {av4.x, av4.y, av4.z, av4.w};
#pragma unroll
      for (int v = 0; v < 4; ++v)
#pragma unroll
        for (int n = 0; n < NO; ++n) O[t][n][v] *= av[v];

      if constexpr (sizeof(TK) == 2) {
        // A = P[node r16][tokens 4*grp..+3]; B = V[tokens 4*grp..+3][dim NO*r16 + n]
        const unsigned p01 = pack_f16x2(pv[0], pv[1]), p23 = pack_f16x2(pv[2], pv[3]);
        const f16x4 A = __builtin_bit_cast(f16x4, uint2{p01, p23});
        const uint2* v2 = (const uint2*)vc;
#pragma unroll
        for (int n = 0; n < NO; ++n)
          O[t][n] = __builtin_amdgcn_mfma_f32_16x16x16f16(A, __builtin_bit_cast(f16x4, v2[n]), O[t][n], 0, 0, 0);
      } else {
        const float* vf = (const float*)vc;
#pragma unroll
        for (int v = 0; v < 4; ++v)
#pragma unroll
          for (int n = 0; n < NO; ++n)
            O[t][n] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[v], vf[n * 4 + v], O[t][n], 0, 0, 0);
      }
    }
  };
  // The paired walk (PAIR, fp16 cache) takes the pages in pairs and keeps
  // two in flight within the registers of one: the first page of a pair
  // arrives in kcur/vcur, the second in the wave's LDS slot (global -> LDS).
  // Once the slot has been read out, the next pair is requested at once (the
  // slot's page first, then the registers' page), so both loads overlap.
  if constexpr (kLdsWalk) {
    if (p + stride < n_pages) dma_page(p + stride, 1);
    __syncthreads();  // q tiles ready
    for (int it = 0; p < n_pages; p += 2 * stride, it += 2) {
      walk_page(p, kcur, vcur);
      if (p + stride >= n_pages) break;
      uint4 ks[NQ], vs[NV];
      asm volatile("" ::: "memory");  // no slot access moves across this point
#pragma unroll
      for (int c = 0; c < NQ; ++c) ks[c] = pslot[c * 64 + lane];
#pragma unroll
      for (int c = 0; c < NV; ++c) vs[c] = pslot[(NQ + c) * 64 + lane];
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the slot is read out before it is refilled
      asm volatile("" ::: "memory");
      if (p + 3 * stride < n_pages) dma_page(p + 3 * stride, it + 3);
      asm volatile("" ::: "memory");
      if (p + 2 * stride < n_pages) load_page(p + 2 * stride, it + 2, kcur, vcur);
      walk_page(p + stride, ks, vs);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // no page load still writes the slot
  } else {
    __syncthreads();  // q tiles ready
    for (int it = 0; p < n_pages; p += stride, ++it) {
      uint4 knext[NQ], vnext[NV];
      if (p + stride < n_pages) load_page(p + stride, it + 1, knext, vnext);
      walk_page(p, kcur, vcur);
#pragma unroll
      for (int c = 0; c < NQ; ++c) kcur[c] = knext[c];
#pragma unroll
      for (int c = 0; c < NV; ++c) vcur[c] = vnext[c];
    }
  }

  // Merge the waves' states tile by tile: O = sum_w f_w O_w / sum_w f_w l_w
  // with f_w = 2^(m_w - max_w m_w), summed in wave order.  Every thread
  // derives the weights of the row it writes from the waves' (m, l) in LDS
  // (the same operations in the same order everywhere), so one barrier
  // separates the waves' writes from the combination.
  float* sm_m = smem + TMAX * 64 * NQ * 4;  // [W][16], after the q tiles
  float* sm_l = sm_m + W * 16;              // [W][16]
  float* sm_o = kLdsWalk ? s_o : sm_l + W * 16;  // [W][64][OS]
  auto row_weights = [&](int row, float (&f)[W]) {
    float mx = -1e30f;
#pragma unroll
    for (int w = 0; w < W; ++w) mx = fmaxf(mx, sm_m[w * 16 + row]);
    float den = 0.f;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      f[w] = exp2f(sm_m[w * 16 + row] - mx);
      den += f[w] * sm_l[w * 16 + row];
    }
    return make_float2(mx, den);
  };
  const size_t slot = ((size_t)head * gridDim.y + y) * a.groups + g;  // this workgroup's partial slot
  // items of several row tiles leave their partial states to k_attn_merge
  // (plain stores: the kernel boundary publishes them)
  const bool defer = a.defer_merge != 0;
  // the partial outputs of the launch: [heads * items * groups][TMAX][16][HD] floats
  const __amdgpu_buffer_rsrc_t pres = __builtin_amdgcn_make_buffer_rsrc(
      a.part_o, (short)0, (int)((size_t)a.n_heads * gridDim.y * a.groups * TMAX * 16 * HD * sizeof(float)), 0x00020000);
#pragma unroll
  for (int t = 0; t < TMAX; ++t) {
    if (t >= T) break;
    if (grp == 0) {
      sm_m[wave * 16 + r16] = m_run[t];
      sm_l[wave * 16 + r16] = l_run[t];
    }
#pragma unroll
    for (int n = 0; n < NO; ++n)
#pragma unroll
      for (int v = 0; v < 4; ++v) sm_o[(wave * 64 + lane) * OS + n * 4 + v] = O[t][n][v];
    __syncthreads();

    // Output (source lane src, row v of its four, tiles n0 .. n0+3): node row
    // 4*(src/16)+v of the tile, dims NO*(src%16)+n0 .. +3 (contiguous, so one
    // vector store each); value sum_w f_w O_w (unnormalised), in wave order.
    static_assert(NO % 4 == 0, "four output tiles per store");
    float* pm = a.part_ml + (slot * TMAX + t) * 32;      // [16][2]
    for (int e = threadIdx.x; e < 64 * NO; e += blockDim.x) {
      const int src = e / NO, v = (e / (NO / 4)) % 4, n0 = (e % (NO / 4)) * 4;
      const int row = (src >> 4) * 4 + v;
      const int ln = t * 16 + row;
      if (ln >= Ms) continue;
      float f[W];
      const float2 md = row_weights(row, f);
      float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int w = 0; w < W; ++w) {
        const float* so = sm_o + (w * 64 + src) * OS + n0 * 4 + v;
        num.x += f[w] * so[0];
        num.y += f[w] * so[4];
        num.z += f[w] * so[8];
        num.w += f[w] * so[12];
      }
      const int dim = NO * (src & 15) + n0;
      if (G == 1) {
        const float den = md.y;
        store_act4<TW>(a.o, a.o_plane, act_index<TW>(row0 + ln, head * HD + dim, a.d),
                       make_float4(num.x / den, num.y / den, num.z / den, num.w / den));
      } else if (defer) {
        *(float4*)(a.part_o + (slot * TMAX + t) * 16 * HD + row * HD + dim) = num;
      } else {
        store_agent4(pres, (int)(((slot * TMAX + t) * 16 * HD + row * HD + dim) * sizeof(float)), num);
      }
    }
    if (G > 1 && threadIdx.x < 16) {
      float f[W];
      const float2 md = row_weights(threadIdx.x, f);
      if (defer) {
        *(float2*)(pm + threadIdx.x * 2) = md;
      } else {
        store_agent(pm + threadIdx.x * 2 + 0, md.x);
        store_agent(pm + threadIdx.x * 2 + 1, md.y);
      }
    }
    __syncthreads();  // the next tile reuses the merge buffers
  }
  if (G == 1 || defer) return;

  // Publish this workgroup's partials, then let the last arrival merge.  Each
  // thread waits until its agent-scope stores are acknowledged (then they are
  // visible to every XCD), the barrier makes that true of the whole
  // workgroup, and only then is the arrival counted; the last arrival reads
  // the partials with agent-scope loads issued after its count returned.
  // (A device-scope fence instead writes back and invalidates this XCD's
  // whole L2.)
  __shared__ int last;
  const int ctr = head * gridDim.y + y;
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0) {
    const int prev = __hip_atomic_fetch_add(a.counters + ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    last = prev == G - 1;
  }
  __syncthreads();
  if (!last) return;
  // Phase 1: per (tile, row) the normalised weight of each partial,
  // w_k = 2^(m_k - max m) / sum_k 2^(m_k - max m) l_k, into LDS (the q tiles
  // are no longer needed).  Phase 2: each thread merges 4 dims of up to R
  // outputs per round (two with several row tiles; one with a single tile,
  // where each thread has one output and the registers stay within what two
  // workgroups per CU allow), reading only the G partials (summed in
  // workgroup order); the first round's loads are issued before phase 1, so
  // the two round trips overlap.
  const size_t slot0 = ((size_t)head * gridDim.y + y) * a.groups;
  float* sm_w = smem;  // [T * 16][kAttnMaxGroups]
  const int n_e4 = T * 4 * HD;
  const size_t part_stride = (size_t)TMAX * 16 * HD;  // floats between consecutive partial slots
  constexpr int R = TMAX >= 2 ? 2 : 1;
  float4 v[R][kAttnMaxGroups];
  auto load_round = [&](int base) {
#pragma unroll
    for (int i = 0; i < R; ++i) {
      // clamped, so every load stays inside the item's partials; the
      // clamped outputs are not stored
      const int e4 = min(base + i * (int)blockDim.x + (int)threadIdx.x, n_e4 - 1);
      const int e = e4 * 4;
      const int t = e / (16 * HD), row = (e / HD) % 16, dim = e % HD;
      const size_t src = (slot0 * TMAX + t) * 16 * HD + row * HD + dim;  // floats
#pragma unroll
      for (int k = 0; k < kAttnMaxGroups; ++k)
        if (k < G) v[i][k] = load_agent4(pres, (int)((src + k * part_stride) * sizeof(float)));
    }
  };
  auto merge_round = [&](int base) {
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const int e4 = base + i * (int)blockDim.x + (int)threadIdx.x;
      if (e4 >= n_e4) continue;
      const int e = e4 * 4;
      const int t = e / (16 * HD), row = (e / HD) % 16, dim = e % HD;
      const int ln = t * 16 + row;
      if (ln >= Ms) continue;
      const float* w = sm_w + (t * 16 + row) * kAttnMaxGroups;
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int k = 0; k < kAttnMaxGroups; ++k) {
        if (k < G) {
          acc.x += w[k] * v[i][k].x;
          acc.y += w[k] * v[i][k].y;
          acc.z += w[k] * v[i][k].z;
          acc.w += w[k] * v[i][k].w;
        }
      }
      store_act4<TW>(a.o, a.o_plane, act_index<TW>(row0 + ln, head * HD + dim, a.d), acc);
    }
  };
  load_round(0);
  for (int idx = threadIdx.x; idx < T * 16; idx += blockDim.x) {
    const int t = idx >> 4, row = idx & 15;
    const float* pm = a.part_ml + (slot0 * TMAX + t) * 32 + row * 2;
    float mk[kAttnMaxGroups], lk[kAttnMaxGroups];
#pragma unroll
    for (int k = 0; k < kAttnMaxGroups; ++k) {
      if (k < G) {
        mk[k] = load_agent(pm + k * TMAX * 32);
        lk[k] = load_agent(pm + k * TMAX * 32 + 1);
      }
    }
    float mx = -1e30f;
#pragma unroll
    for (int k = 0; k < kAttnMaxGroups; ++k)
      if (k < G) mx = fmaxf(mx, mk[k]);
    float f[kAttnMaxGroups], den = 0.f;
#pragma unroll
    for (int k = 0; k < kAttnMaxGroups; ++k) {
      f[k] = k < G ? exp2f(mk[k] - mx) : 0.f;
      if (k < G) den += f[k] * lk[k];
    }
    const float inv = 1.f / den;
#pragma unroll
    for (int k = 0; k < kAttnMaxGroups; ++k) sm_w[idx * kAttnMaxGroups + k] = f[k] * inv;
  }
  __syncthreads();
  merge_round(0);
  for (int base = R * (int)blockDim.x; base < n_e4; base += R * (int)blockDim.x) {
    load_round(base);
    merge_round(base);
  }
  if (threadIdx.x == 0) a.counters[ctr] = 0;
}

// The deferred merge: workgroup (head, item, z) combines rows 8 z .. 8 z + 7
// of the item from its G partial states (plain loads: the attention launch
// has ended), one thread per four adjacent dimensions of a row, summed in
// workgroup order; items the attention launch finished itself (G = 1) are
// skipped.
constexpr int kMergeRows = 8;
template <typename TW, int HD, int TMAX>
__global__ __launch_bounds__(kMergeRows * HD / 4) void k_attn_merge(AttnArgs a) {
  const int head = blockIdx.x, y = blockIdx.y, z = blockIdx.z;
  const int row0 = a.item_row0[y], Ms = a.item_rows[y];
  const int lr = z * kMergeRows + (int)threadIdx.x / (HD / 4);  // row of the item
  if (lr >= Ms) return;
  const int T = (Ms + 15) >> 4;
  const int G = attn_item_groups(a, (a.sp->seq_nkv[a.item_seg[y]] + a.item_slots[y] + kPage - 1) / kPage, T);
  if (G == 1) return;
  const int dim = ((int)threadIdx.x % (HD / 4)) * 4;
  const int t = lr >> 4, row = lr & 15;
  const size_t slot0 = ((size_t)head * gridDim.y + y) * a.groups;
  float2 ml[kAttnMaxGroups];
  float4 o[kAttnMaxGroups];
#pragma unroll
  for (int k = 0; k < kAttnMaxGroups; ++k) {
    if (k < G) {
      const size_t sl = (slot0 + k) * TMAX + t;
      ml[k] = *(const float2*)(a.part_ml + sl * 32 + row * 2);
      o[k] = *(const float4*)(a.part_o + sl * 16 * HD + row * HD + dim);
    }
  }
  float mx = -1e30f;
#pragma unroll
  for (int k = 0; k < kAttnMaxGroups; ++k)
    if (k < G) mx = fmaxf(mx, ml[k].x);
  float den = 0.f;
  float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int k = 0; k < kAttnMaxGroups; ++k) {
    if (k < G) {
      const float f = exp2f(ml[k].x - mx);
      den += f * ml[k].y;
      num.x += f * o[k].x;
      num.y += f * o[k].y;
      num.z += f * o[k].z;
      num.w += f * o[k].w;
    }
  }
  store_act4<TW>(a.o, a.o_plane, act_index<TW>(row0 + lr, head * HD + dim, a.d),
                 make_float4(num.x / den, num.y / den, num.z / den, num.w / den));
}

template <typename TK, typename TW, int HD, int TMAX>
static hipError_t attn_attr() {
  hipError_t e = hipFuncSetAttribute((const void*)k_attn<TK, TW, HD, TMAX, false>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)attn_lds<TK, HD, TMAX, false>());
  if constexpr (sizeof(TK) == 2)
    if (e == hipSuccess)
      e = hipFuncSetAttribute((const void*)k_attn<TK, TW, HD, TMAX, true>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)attn_lds<TK, HD, TMAX, true>());
  return e;
}

template <typename TK, typename TW, int HD>
static hipError_t attn_attr_hd() {
  hipError_t e = attn_attr<TK, TW, HD, 1>();
  if (e == hipSuccess) e = attn_attr<TK, TW, HD, 2>();
  if (e == hipSuccess) e = attn_attr<TK, TW, HD, 4>();
  return e;
}

// Raises the LDS limit of the attention kernels (more than 64 KiB); done once
// at context creation so that no attribute call falls inside a captured step.
hipError_t init_kernel_attributes() {
  hipError_t e = attn_attr_hd<_Float16, _Float16, 128>();
  if (e == hipSuccess) e = attn_attr_hd<_Float16, _Float16, 64>();
  if (e == hipSuccess) e = attn_attr_hd<float, float, 128>();
  if (e == hipSuccess) e = attn_attr_hd<float, float, 64>();
  return e;
}

template <typename TK, typename TW, int HD, int TMAX>
static hipError_t attn_t(int n_seq, const AttnArgs& a, hipStream_t s) {
  constexpr size_t lds_one = attn_lds<TK, HD, TMAX, false>();
  bool launched = false;
  if constexpr (sizeof(TK) == 2) {
    if (a.pages_per_wg == 0) {  // one KV sequence: the paired walk
      constexpr size_t lds_pair = attn_lds<TK, HD, TMAX, true>();
      TSS_LAUNCH((k_attn<TK, TW, HD, TMAX, true>), dim3(a.n_heads, n_seq, a.groups), dim3(kAttnWaves * 64),
                 lds_pair, s, a);
      launched = true;
    }
  }
  if (!launched)
    TSS_LAUNCH((k_attn<TK, TW, HD, TMAX, false>), dim3(a.n_heads, n_seq, a.groups), dim3(kAttnWaves * 64), lds_one,
               s, a);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess && a.defer_merge) {
    TSS_LAUNCH((k_attn_merge<TW, HD, TMAX>), dim3(a.n_heads, n_seq, TMAX * 16 / kMergeRows),
               dim3(kMergeRows * HD / 4), 0, s, a);
    e = hipGetLastError();
  }
  return e;
}

template <typename TK, typename TW, int HD>
static hipError_t attn_hd(int tiles, int n_seq, const AttnArgs& a, hipStream_t s) {
  if (tiles <= 1) return attn_t<TK, TW, HD, 1>(n_seq, a, s);
  if (tiles <= 2) return attn_t<TK, TW, HD, 2>(n_seq, a, s);
  return attn_t<TK, TW, HD, 4>(n_seq, a, s);
}

// max_tiles = most 16-row tiles of an item (1..4); n_seq = items (grid.y).
hipError_t launch_attn(bool bf16, int head_dim, int max_tiles, int n_seq, const AttnArgs& a, hipStream_t s) {
  if (max_tiles < 1 || max_tiles > 4 || n_seq < 1 || n_seq > kAttnMaxItems) return hipErrorInvalidValue;
  if (bf16)
    return head_dim == 128 ? attn_hd<_Float16, _Float16, 128>(max_tiles, n_seq, a, s)
                           : attn_hd<_Float16, _Float16, 64>(max_tiles, n_seq, a, s);
  return head_dim == 128 ? attn_hd<float, float, 128>(max_tiles, n_seq, a, s)
                         : attn_hd<float, float, 64>(max_tiles, n_seq, a, s);
}

}  // namespace tss
