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

// One workgroup of 16 waves.  Greedy token per row from the lm_head's
// per-strip partials (each row gets 16 / M waves, loads issued eight at a
// time), then one accept scan per sequence over its tree: a node is accepted
// when its parent is and its token equals the parent's greedy token; the
// deepest accepted node (lowest id among equal depths) gives accept_len and
// the bonus token.
__global__ __launch_bounds__(1024) void k_accept(AcceptArgs a) {
  __shared__ int32_t g[kMaxRows];
  __shared__ float bvs[16];
  __shared__ int32_t bis[16];
  __shared__ int32_t s_tok[kMaxRows];
  __shared__ int8_t s_par[kMaxRows];
  __shared__ uint8_t s_dep[kMaxRows];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int M = a.M;
  if (threadIdx.x < M) {
    s_tok[threadIdx.x] = a.sp->tok[threadIdx.x];
    s_par[threadIdx.x] = a.sp->parent[threadIdx.x];
    s_dep[threadIdx.x] = a.sp->depth[threadIdx.x];
  }
  const int wpr = M >= 16 ? 1 : (M >= 8 ? 2 : (M >= 4 ? 4 : (M >= 2 ? 8 : 16)));  // waves per row
  const int groups = 16 / wpr;
  const int grp_id = wave / wpr, sub = wave % wpr;
  for (int m0 = 0; m0 < M; m0 += groups) {
    const int m = m0 + grp_id;
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    if (m < M) {
      const int stride = 64 * wpr;
      for (int p = sub * 64 + lane; p < a.nparts; p += 8 * stride) {
        float v[8];
        int ix[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int q = p + u * stride;
          v[u] = q < a.nparts ? a.am_val[(size_t)m * a.am_stride + q] : -INFINITY;
          ix[u] = q < a.nparts ? a.am_idx[(size_t)m * a.am_stride + q] : 0x7fffffff;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (better(v[u], ix[u], bv, bi)) { bv = v[u]; bi = ix[u]; }
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const float ov = __shfl_xor(bv, off);
      const int oi = __shfl_xor(bi, off);
      if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    if (lane == 0) {
      bvs[wave] = bv;
      bis[wave] = bi;
    }
    __syncthreads();
    if (sub == 0 && lane == 0 && m < M) {
      for (int w = 1; w < wpr; ++w)
        if (better(bvs[wave + w], bis[wave + w], bv, bi)) { bv = bvs[wave + w]; bi = bis[wave + w]; }
      g[m] = bi;
      a.greedy[m] = bi;
    }
    __syncthreads();
  }
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
  TSS_LAUNCH(k_accept, dim3(1), dim3(1024), 0, s, a);
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
