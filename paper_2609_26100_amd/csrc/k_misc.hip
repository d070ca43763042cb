// Small kernels around the projections and attention of the verify step:
// embedding gather, greedy argmax + accept scan, tree-path KV compaction and
// the rotary cos/sin table.
#include "tss_internal.h"

namespace tss {

// h[m] = E[tok[m]] (fp32); xn[m] = h[m] * gain (activation planes) for the
// first RMSNorm the rows meet; ss_out[m] = sum h[m]^2 (one partial,
// fixed-order reduction).
template <typename T>
__global__ __launch_bounds__(256) void k_embed(EmbedArgs a) {
  __shared__ float red[256];
  const int m = blockIdx.x;
  const int d = a.d;
  const T* row = (const T*)a.embed + (size_t)a.sp->tok[m] * d;
  float s = 0.f;
  for (int k = threadIdx.x; k < d; k += 256) {
    const float v = (float)row[k];
    a.h[(size_t)m * d + k] = v;
    store_act<T>(a.xn, a.xn_plane, (size_t)m * d + k, v * a.gain[k]);
    s += v * v;
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (threadIdx.x < off) red[threadIdx.x] += red[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) a.ss_out[m] = red[0];
}

// (value, index) order of the greedy argmax: larger value first, lower index on ties.
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

// One workgroup.  Greedy token per node from the lm_head's per-strip partials,
// then the accept scan over the tree: a node is accepted when its parent is
// and its token equals the parent's greedy token; the deepest accepted node
// (lowest id among equal depths) gives accept_len and the bonus token.
__global__ __launch_bounds__(256) void k_accept(AcceptArgs a) {
  __shared__ int32_t g[kMaxNodes];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int m = wave; m < a.M; m += 4) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    for (int p = lane; p < a.nparts; p += 64) {
      const float v = a.am_val[(size_t)p * a.Mp + m];
      const int i = a.am_idx[(size_t)p * a.Mp + m];
      if (better(v, i, bv, bi)) { bv = v; bi = i; }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const float ov = __shfl_xor(bv, off);
      const int oi = __shfl_xor(bi, off);
      if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    if (lane == 0) {
      g[m] = bi;
      a.greedy[m] = bi;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const StepParams* sp = a.sp;
    uint64_t acc = 1ull;  // bit i: node i accepted
    int best = 0;
    for (int i = 1; i < a.M; ++i) {
      const int p = sp->parent[i];
      if (((acc >> p) & 1ull) && sp->tok[i] == g[p]) {
        acc |= 1ull << i;
        if (sp->depth[i] > sp->depth[best]) best = i;
      }
    }
    Result* r = a.result;
    const int len = sp->depth[best];
    r->accept_len = len;
    r->next_token = g[best];
    r->best = best;
    r->path_len = len + 1;
    for (int j = best, dd = len; dd >= 0; --dd) {
      r->path[dd] = j;
      j = dd > 0 ? sp->parent[j] : 0;
    }
  }
}

// Moves the K/V of the accepted tree path (nodes path[1..a]) to the slots
// right after the context (n_kv + 1 .. n_kv + a), for the layers that ran.
// Every source slot n_kv + path[d] has path[d] >= d, so reading all sources
// before writing any destination is enough; one thread owns one dimension.
// T = KV element type.
template <typename T>
__global__ __launch_bounds__(128) void k_compact(CompactArgs a) {
  const int layer = blockIdx.x, head = blockIdx.y, dim = threadIdx.x;
  if (a.sp->mask[layer] || dim >= a.head_dim) return;
  const int len = a.result->accept_len;
  const int HD = a.head_dim;
  T kbuf[kMaxNodes], vbuf[kMaxNodes];
  auto kaddr = [&](int slot) {
    const int page = a.page_table[slot >> 4], tin = slot & 15;
    T* blk = (T*)a.kv_pages + ((((size_t)layer * a.n_pages_pool + page) * 2 + 0) * a.n_heads + head) * (16 * (size_t)HD);
    return blk + tin * HD + dim;
  };
  auto vaddr = [&](int slot) {
    const int page = a.page_table[slot >> 4], tin = slot & 15;
    T* blk = (T*)a.kv_pages + ((((size_t)layer * a.n_pages_pool + page) * 2 + 1) * a.n_heads + head) * (16 * (size_t)HD);
    return blk + (tin >> 2) * HD * 4 + dim * 4 + (tin & 3);
  };
  for (int d = 1; d <= len; ++d) {
    const int src = a.n_kv + a.result->path[d];
    kbuf[d] = *kaddr(src);
    vbuf[d] = *vaddr(src);
  }
  for (int d = 1; d <= len; ++d) {
    if (a.result->path[d] == d) continue;
    *kaddr(a.n_kv + d) = kbuf[d];
    *vaddr(a.n_kv + d) = vbuf[d];
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

hipError_t launch_embed(bool bf16, const EmbedArgs& a, hipStream_t s) {
  if (bf16)
    hipLaunchKernelGGL(k_embed<__bf16>, dim3(a.M), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(k_embed<float>, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_accept(const AcceptArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_accept, dim3(1), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_compact(bool bf16, const CompactArgs& a, hipStream_t s) {
  if (bf16)
    hipLaunchKernelGGL(k_compact<_Float16>, dim3(a.n_layers, a.n_heads), dim3(128), 0, s, a);
  else
    hipLaunchKernelGGL(k_compact<float>, dim3(a.n_layers, a.n_heads), dim3(128), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_rope_table(float2* tab, int max_pos, int head_dim, float base, hipStream_t s) {
  const int n = max_pos * (head_dim >> 1);
  hipLaunchKernelGGL(k_rope_table, dim3((n + 255) / 256), dim3(256), 0, s, tab, max_pos, head_dim, base);
  return hipGetLastError();
}

}  // namespace tss
