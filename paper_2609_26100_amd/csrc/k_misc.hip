// Small kernels around the projections and attention of the verify step:
// embedding gather, greedy argmax + accept scan, tree-path KV compaction and
// the rotary cos/sin table.
#include "tss_internal.h"

namespace tss {

// h[m] = E[tok[m]] (fp32), or a saved residual row (src_h); xn[m] = h[m] * gain (activation planes) with the
// gain of the first RMSNorm the row's sequence meets; ss_out[m][p] = sum of
// h[m][k]^2 over the 16 columns of part p (the format every projection
// epilogue writes, so each norm reads d/16 parts whatever produced them).
// The step's parameters arrive by value and workgroup 0 stores them for the
// later kernels of the step (this replaces a separate host-to-device copy,
// which costs as much as a kernel launch).
template <typename T>
__global__ __launch_bounds__(256) void k_embed(EmbedArgs a) {
  constexpr int E = 16 / (int)sizeof(T);  // elements of T per 16-byte chunk
  const int m = blockIdx.x;
  const int d = a.d;
  if (m == 0) {
    const uint32_t* src = (const uint32_t*)&a.sp;
    uint32_t* dst = (uint32_t*)a.sp_dev;
    for (int i = threadIdx.x; i < (int)(sizeof(StepParams) / 4); i += 256) dst[i] = src[i];
    // a step whose blocks are all skipped reports no attention items
    if (threadIdx.x == 0) a.attn_split[2 * kAttnMaxItems] = 0;
    // the merges' arrival counters start every step at zero (their last
    // arrivals also reset them; this holds even when another context's step
    // used the same memory in between)
    for (int i = threadIdx.x; i < a.n_counters; i += 256) a.counters[i] = 0;
  }
  const float* gain = a.gain[a.sp.row_seq[m]];
  // Each thread takes whole 16-column parts (up to two; d <= 8192): the
  // row's chunks and the gains of its parts are requested together, and the
  // part's sum of squares needs no exchange between threads.  The row is the
  // token's embedding (T) or a saved residual row (fp32).
  const bool resume = a.src_h != nullptr;
  const int CPP = resume ? 4 : 16 / E;  // 16-byte chunks per part
  const uint4* row = resume ? (const uint4*)(a.src_h + (size_t)(m - a.sp.seq_row0[a.sp.row_seq[m]]) * d)
                            : (const uint4*)((const T*)a.embed + (size_t)a.sp.tok[m] * d);
  const int nparts = d / 16;
  uint4 raw[2][4];
  float4 gv[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int p = threadIdx.x + 256 * i;
    if (p >= nparts) break;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (j < CPP) raw[i][j] = row[p * CPP + j];
#pragma unroll
    for (int q = 0; q < 4; ++q) gv[i][q] = ((const float4*)gain)[p * 4 + q];
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int p = threadIdx.x + 256 * i;
    if (p >= nparts) break;
    float v[16];
    if (resume) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 f = __builtin_bit_cast(float4, raw[i][j]);
        v[4 * j] = f.x;
        v[4 * j + 1] = f.y;
        v[4 * j + 2] = f.z;
        v[4 * j + 3] = f.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < 16 / E; ++j) {
        const T* e = (const T*)&raw[i][j];
#pragma unroll
        for (int k = 0; k < E; ++k) v[j * E + k] = (float)e[k];
      }
    }
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) ss += v[k] * v[k];
    float* hrow = a.h + (size_t)m * d + p * 16;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 h4 = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
      *(float4*)(hrow + 4 * q) = h4;
      const float4 g4 = gv[i][q];
      store_act4<T>(a.xn, a.xn_plane, act_index<T>(m, p * 16 + 4 * q, d),
                    make_float4(h4.x * g4.x, h4.y * g4.y, h4.z * g4.z, h4.w * g4.w));
    }
    a.ss_out[(size_t)m * a.ss_stride + p] = ss;
  }
}

// (value, index) order of the greedy argmax: larger value first, lower index on ties.
// NaN counts as the largest value (the lowest index among NaNs), as numpy's
// argmax has it, so a row with NaN logits still yields an in-range token.
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  const bool nv = __builtin_isnan(v), nb = __builtin_isnan(bv);
  return (nv && !nb) || v > bv || ((v == bv || (nv && nb)) && i < bi);
}

// Greedy token per row, one workgroup of 256 threads per row: each thread
// reduces its share of the lm_head's per-strip (max, argmax) partials (all of
// its loads issued together), then the wave and the workgroup combine theirs
// in a fixed order (the order of `better` is total, so the result does not
// depend on it anyway).  The rows' greedy tokens are published with
// agent-scope stores; the last workgroup to arrive (a counter bumped after
// the store has landed) runs one accept scan per sequence over its tree: a
// node is accepted when its parent is and its token equals the parent's
// greedy token; the deepest accepted node (lowest id among equal depths)
// gives accept_len and the bonus token.
constexpr int kAcceptThreads = 256;
constexpr int kAcceptLoads = 8;  // partials per thread per round (2048 per round: V = 32000 in one)
__global__ __launch_bounds__(kAcceptThreads) void k_accept(AcceptArgs a) {
  __shared__ float bvs[kAcceptThreads / 64];
  __shared__ int32_t bis[kAcceptThreads / 64];
  __shared__ int last;
  __shared__ int32_t g[kMaxRows];
  __shared__ int32_t s_tok[kMaxRows];
  __shared__ int8_t s_par[kMaxRows];
  __shared__ uint8_t s_dep[kMaxRows];
  const int m = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  // the row's partials through buffer resources: loads past the row return
  // zeros (replaced below), so none needs a branch
  const __amdgpu_buffer_rsrc_t vres = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.am_val + (size_t)m * a.am_stride), (short)0, a.nparts * 4, 0x00020000);
  const __amdgpu_buffer_rsrc_t ires = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.am_idx + (size_t)m * a.am_stride), (short)0, a.nparts * 4, 0x00020000);
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int p0 = threadIdx.x; p0 < a.nparts; p0 += kAcceptLoads * kAcceptThreads) {
    float v[kAcceptLoads];
    int ix[kAcceptLoads];
#pragma unroll
    for (int u = 0; u < kAcceptLoads; ++u) {
      const int q = p0 + u * kAcceptThreads;
      v[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(vres, q * 4, 0, 0));
      ix[u] = (int)__builtin_amdgcn_raw_buffer_load_b32(ires, q * 4, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < kAcceptLoads; ++u) {
      const bool in = p0 + u * kAcceptThreads < a.nparts;
      if (in && better(v[u], ix[u], bv, bi)) {
        bv = v[u];
        bi = ix[u];
      }
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(bv, off);
    const int oi = __shfl_xor(bi, off);
    if (better(ov, oi, bv, bi)) {
      bv = ov;
      bi = oi;
    }
  }
  if (lane == 0) {
    bvs[wave] = bv;
    bis[wave] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kAcceptThreads / 64; ++w)
      if (better(bvs[w], bis[w], bv, bi)) {
        bv = bvs[w];
        bi = bis[w];
      }
    __hip_atomic_store(a.greedy + m, bi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    last = __hip_atomic_fetch_add(a.count, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (int)gridDim.x - 1;
  }
  __syncthreads();
  if (!last) return;

  const int M = a.M;
  for (int i = threadIdx.x; i < M; i += kAcceptThreads) {
    g[i] = __hip_atomic_load(a.greedy + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_tok[i] = a.sp->tok[i];
    s_par[i] = a.sp->parent[i];
    s_dep[i] = a.sp->depth[i];
  }
  __syncthreads();
  const int sq = threadIdx.x;
  if (sq < a.sp->n_seqs) {
    const int r0 = a.sp->seq_row0[sq], n = a.sp->seq_row0[sq + 1] - r0;
    const int32_t* gs = g + r0;
    uint64_t acc = 1ull;  // bit i: local node i accepted
    int best = 0;
    for (int i = 1; i < n; ++i) {
      const int p = s_par[r0 + i];
      if (((acc >> p) & 1ull) && s_tok[r0 + i] == gs[p]) {
        acc |= 1ull << i;
        if (s_dep[r0 + i] > s_dep[r0 + best]) best = i;
      }
    }
    const int len = s_dep[r0 + best];
    for (int copy = 0; copy < 2; ++copy) {
      Result* r = (copy == 0 ? a.result : a.result_host) + sq;
      r->accept_len = len;
      r->next_token = gs[best];
      r->best = best;
      r->path_len = len + 1;
      for (int j = best, dd = len; dd >= 0; --dd) {
        r->path[dd] = j;
        j = dd > 0 ? s_par[r0 + j] : 0;
      }
    }
  }
  if (threadIdx.x == 0) *a.count = 0;
}

// Moves the K/V of an accepted tree path (local nodes path[1..a]) to the
// slots right after the context (n_kv + 1 .. n_kv + a), for the layers its
// sequence ran.  Every source slot n_kv + path[d] has path[d] >= d, so
// reading all sources before writing any destination is enough; one thread
// owns one dimension.  grid = (layer, head, listed sequence); T = KV type.
template <typename T>
__global__ __launch_bounds__(128) void k_compact(CompactArgs a) {
  const int layer = blockIdx.x, head = blockIdx.y, z = blockIdx.z, dim = threadIdx.x;
  if (!((a.lay_on[z][layer >> 6] >> (layer & 63)) & 1ull) || dim >= a.head_dim) return;
  const int sq = a.seq[z];
  const int n_kv = a.sp->seq_nkv[sq];
  const Result& res = a.result[sq];
  const int len = res.accept_len;
  const int HD = a.head_dim;
  const int32_t* pt = a.page_table + a.pt_off[z];
  T kbuf[kMaxNodes], vbuf[kMaxNodes];
  auto kaddr = [&](int slot) {
    const int page = pt[slot >> 4], tin = slot & 15;
    T* blk = (T*)a.kv_pages + ((((size_t)layer * a.n_pages_pool + page) * 2 + 0) * a.n_heads + head) * (16 * (size_t)HD);
    return blk + tin * HD + dim;
  };
  auto vaddr = [&](int slot) {
    const int page = pt[slot >> 4], tin = slot & 15;
    T* blk = (T*)a.kv_pages + ((((size_t)layer * a.n_pages_pool + page) * 2 + 1) * a.n_heads + head) * (16 * (size_t)HD);
    return blk + (tin >> 2) * HD * 4 + dim * 4 + (tin & 3);
  };
  for (int d = 1; d <= len; ++d) {
    const int src = n_kv + res.path[d];
    kbuf[d] = *kaddr(src);
    vbuf[d] = *vaddr(src);
  }
  for (int d = 1; d <= len; ++d) {
    if (res.path[d] == d) continue;
    *kaddr(n_kv + d) = kbuf[d];
    *vaddr(n_kv + d) = vbuf[d];
  }
}

// tab[pos][j] = (cos, sin)(pos * base^(-2j/hd)), formed in double precision.
__global__ void k_rope_table(float2* tab, int max_pos, int head_dim, float base) {
  const int half = head_dim >> 1;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= max_pos * half) return;
  const int pos = i / half, j = i % half;
  const double inv = pow((double)base, -2.0 * (double)j / (double)head_dim);
  const double ang = (double)pos * inv;
  tab[i] = make_float2((float)cos(ang), (float)sin(ang));
}

const void* embed_kernel(bool bf16) {
  return bf16 ? (const void*)k_embed<_Float16> : (const void*)k_embed<float>;
}

hipError_t launch_embed(bool bf16, const EmbedArgs& a, hipStream_t s) {
  if (bf16)
    TSS_LAUNCH(k_embed<_Float16>, dim3(a.M), dim3(256), 0, s, a);
  else
    TSS_LAUNCH(k_embed<float>, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_accept(const AcceptArgs& a, hipStream_t s) {
  if (a.M < 1 || a.M > kMaxRows || !a.count) return hipErrorInvalidValue;
  TSS_LAUNCH(k_accept, dim3(a.M), dim3(kAcceptThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_compact(bool bf16, int n_seqs, const CompactArgs& a, hipStream_t s) {
  if (bf16)
    TSS_LAUNCH(k_compact<_Float16>, dim3(a.n_layers, a.n_heads, n_seqs), dim3(128), 0, s, a);
  else
    TSS_LAUNCH(k_compact<float>, dim3(a.n_layers, a.n_heads, n_seqs), dim3(128), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_rope_table(float2* tab, int max_pos, int head_dim, float base, hipStream_t s) {
  const int n = max_pos * (head_dim >> 1);
  TSS_LAUNCH(k_rope_table, dim3((n + 255) / 256), dim3(256), 0, s, tab, max_pos, head_dim, base);
  return hipGetLastError();
}

}  // namespace tss
