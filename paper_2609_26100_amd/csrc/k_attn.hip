// Tree-masked attention of the verify step over the paged KV cache (gfx950).
//
// For every head and node i: softmax(q_i K^T / sqrt(hd)) V over the cached
// context [0, n_kv) plus the draft nodes visible to i (i itself and its
// ancestors; their K/V were appended at slots n_kv + j by the QKV kernel).
// This is the attention half of an active block; bypassed blocks never reach
// this kernel (Domain-Aware Skip Controller, block rule).
//
// G workgroups of 16 waves share (head, 16-node tile); wave w of workgroup g
// walks pages 16 g + w, 16 (g + G) + w, ..., loading the next page while it
// computes the current one:
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
// The 16 waves' softmax states meet in LDS (fixed order).  With G = 1 the
// workgroup writes the normalised rows itself.  With G > 1 each workgroup
// writes its partial state, releases it, and bumps a per-(head, tile)
// counter; the last to arrive merges the G partials in workgroup order and
// resets the counter.  No second kernel (a kernel boundary costs about 3 us
// on this GPU) and bit-reproducible results.
#include "tss_internal.h"

namespace tss {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ unsigned pack_f16x2(float lo, float hi) {
  const _Float16 a = (_Float16)lo, b = (_Float16)hi;
  return (unsigned)__builtin_bit_cast(unsigned short, a) | ((unsigned)__builtin_bit_cast(unsigned short, b) << 16);
}

constexpr int kAttnWaves = 16;

// TK = KV element type (_Float16 or float); TW = weight type of the mode
// (selects the activation plane format of the output).
template <typename TK, typename TW, int HD>
__global__ __launch_bounds__(kAttnWaves * 64) void k_attn(AttnArgs a) {
  constexpr int DL = HD / 4;                         // dims per lane group in Q K^T
  constexpr int NQ = DL * (int)sizeof(TK) / 16;      // 16-byte K/Q chunks per lane
  constexpr int NO = HD / 16;                        // output tiles of P V
  constexpr int NV = NO * 4 * (int)sizeof(TK) / 16;  // 16-byte V chunks per lane
  constexpr int W = kAttnWaves;

  const int head = blockIdx.x, qt = blockIdx.y, g = blockIdx.z, G = gridDim.z;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, r16 = lane & 15, grp = lane >> 4;
  // this tile's rows and their sequence: nodes row0 .. row0 + rows - 1 are
  // local nodes j0 .. of a sequence with Ms nodes and n_kv cached tokens
  const int sq = a.tile_seq[qt], row0 = a.tile_row0[qt], rows = a.tile_rows[qt];
  const int n_kv = a.sp->seq_nkv[sq];
  const int Ms = a.sp->seq_row0[sq + 1] - a.sp->seq_row0[sq];
  const int qn = row0 + r16;
  const bool row_ok = r16 < rows;
  const int32_t* pt = a.page_table + a.pt_off[sq];
  const int arg_pages = sq == 0 ? a.n_arg_pages : 0;

  // B operand of S = K Q^T: lane (node qn, group grp) holds q[qn][head*HD + grp*DL + 0..DL).
  // Every wave uses the same tile, so wave 0 builds it once in LDS and the
  // waves read it back per page instead of holding it in registers.
  extern __shared__ float smem[];
  uint4* sm_q = (uint4*)smem;              // [64][NQ]
  if (wave == 0) {
    const float* qrow = a.q + (size_t)qn * a.d + head * HD + grp * DL;
#pragma unroll
    for (int c = 0; c < NQ; ++c) {
      uint4 qv = uint4{0, 0, 0, 0};
      if (row_ok) {
        if constexpr (sizeof(TK) == 2) {
          const float4 f0 = *(const float4*)(qrow + c * 8);
          const float4 f1 = *(const float4*)(qrow + c * 8 + 4);
          qv = uint4{pack_f16x2(f0.x, f0.y), pack_f16x2(f0.z, f0.w), pack_f16x2(f1.x, f1.y), pack_f16x2(f1.z, f1.w)};
        } else {
          qv = *(const uint4*)(qrow + c * 4);
        }
      }
      sm_q[lane * NQ + c] = qv;
    }
  }
  const uint64_t anc = row_ok ? a.sp->anc[qn] : 0ull;
  const int n_pages = (n_kv + Ms + kPage - 1) / kPage;

  float m_run = -1e30f, l_run = 0.f;
  f32x4 O[NO];
#pragma unroll
  for (int n = 0; n < NO; ++n) O[n] = f32x4{0.f, 0.f, 0.f, 0.f};

  const size_t blk_elems = 16 * (size_t)HD;
  auto load_page = [&](int p, uint4 (&kreg)[NQ], uint4 (&vreg)[NV]) {
    const int phys = p < arg_pages ? a.pages[p] : pt[p];  // p is uniform across the wave
    const TK* kb = (const TK*)a.kv_pages + (((size_t)a.layer * a.n_pages_pool + phys) * 2 * a.n_heads + head) * blk_elems;
    const TK* vb = kb + (size_t)a.n_heads * blk_elems;
    const uint4* kp = (const uint4*)(kb + r16 * HD + grp * DL);
    const uint4* vp = (const uint4*)(vb + grp * HD * 4 + r16 * NO * 4);
#pragma unroll
    for (int c = 0; c < NQ; ++c) kreg[c] = kp[c];
#pragma unroll
    for (int c = 0; c < NV; ++c) vreg[c] = vp[c];
  };

  uint4 kcur[NQ], vcur[NV];
  const int stride = W * G;
  int p = g * W + wave;
  if (p < n_pages) load_page(p, kcur, vcur);
  __syncthreads();  // q tile ready
  for (; p < n_pages; p += stride) {
    uint4 knext[NQ], vnext[NV];
    if (p + stride < n_pages) load_page(p + stride, knext, vnext);

    f32x4 S = f32x4{0.f, 0.f, 0.f, 0.f};
    asm volatile("" ::: "memory");  // re-read the q tile from LDS each page (keeps it out of registers)
#pragma unroll
    for (int c = 0; c < NQ; ++c) {
      const uint4 qv = sm_q[lane * NQ + c];
      if constexpr (sizeof(TK) == 2) {
        S = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, kcur[c]),
                                                   __builtin_bit_cast(f16x8, qv), S, 0, 0, 0);
      } else {
        S = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kcur[c].x), __uint_as_float(qv.x), S, 0, 0, 0);
        S = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kcur[c].y), __uint_as_float(qv.y), S, 0, 0, 0);
        S = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kcur[c].z), __uint_as_float(qv.z), S, 0, 0, 0);
        S = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kcur[c].w), __uint_as_float(qv.w), S, 0, 0, 0);
      }
    }

    // S[v] = score of token 4*grp+v of this page against node qn.
    float s[4];
    float mloc = -INFINITY;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int slot = p * kPage + grp * 4 + v;
      bool vis;
      if (slot < n_kv) {
        vis = true;
      } else {
        const int j = slot - n_kv;
        vis = j < Ms && ((anc >> j) & 1ull);
      }
      s[v] = vis ? S[v] * a.scale_log2 : -INFINITY;
      mloc = fmaxf(mloc, s[v]);
    }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float m_new = fmaxf(m_run, mloc);
    const float alpha = exp2f(m_run - m_new);
    float pv[4];
    float lsum = 0.f;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      pv[v] = exp2f(s[v] - m_new);
      lsum += pv[v];
    }
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);
    l_run = l_run * alpha + lsum;
    m_run = m_new;

    // O rows are nodes 4*grp+v; their rescale factor lives in lane 4*grp+v.
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const float av = __shfl(alpha, grp * 4 + v);
#pragma unroll
      for (int n = 0; n < NO; ++n) O[n][v] *= av;
    }

    if constexpr (sizeof(TK) == 2) {
      // A = P[node r16][tokens 4*grp..+3]; B = V[tokens 4*grp..+3][dim NO*r16 + n]
      const unsigned p01 = pack_f16x2(pv[0], pv[1]), p23 = pack_f16x2(pv[2], pv[3]);
      const f16x4 A = __builtin_bit_cast(f16x4, uint2{p01, p23});
      const uint2* v2 = (const uint2*)vcur;
#pragma unroll
      for (int n = 0; n < NO; ++n)
        O[n] = __builtin_amdgcn_mfma_f32_16x16x16f16(A, __builtin_bit_cast(f16x4, v2[n]), O[n], 0, 0, 0);
    } else {
      const float* vf = (const float*)vcur;
#pragma unroll
      for (int v = 0; v < 4; ++v)
#pragma unroll
        for (int n = 0; n < NO; ++n)
          O[n] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[v], vf[n * 4 + v], O[n], 0, 0, 0);
    }
#pragma unroll
    for (int c = 0; c < NQ; ++c) kcur[c] = knext[c];
#pragma unroll
    for (int c = 0; c < NV; ++c) vcur[c] = vnext[c];
  }

  // Merge the waves' states: O = sum_w f_w O_w / sum_w f_w l_w with
  // f_w = 2^(m_w - max_w m_w), summed in wave order.
  constexpr int OS = NO * 4 + 1;
  float* sm_m = smem + 64 * NQ * 4;       // [W][16], after the q tile
  float* sm_l = sm_m + W * 16;            // [W][16]
  float* sm_o = sm_l + W * 16;            // [W][64][OS]
  if (grp == 0) {
    sm_m[wave * 16 + r16] = m_run;
    sm_l[wave * 16 + r16] = l_run;
  }
#pragma unroll
  for (int n = 0; n < NO; ++n)
#pragma unroll
    for (int v = 0; v < 4; ++v) sm_o[(wave * 64 + lane) * OS + n * 4 + v] = O[n][v];
  __syncthreads();

  // Row factors once: mx = max_w m_w, f_w = 2^(m_w - mx), den = sum_w f_w l_w.
  float* sm_mx = sm_o + W * 64 * OS;      // [16]
  float* sm_f = sm_mx + 16;               // [W][16]
  float* sm_den = sm_f + W * 16;          // [16]
  if (threadIdx.x < 16) {
    float mx = -1e30f;
    for (int w = 0; w < W; ++w) mx = fmaxf(mx, sm_m[w * 16 + threadIdx.x]);
    sm_mx[threadIdx.x] = mx;
  }
  __syncthreads();
  if (threadIdx.x < W * 16) sm_f[threadIdx.x] = exp2f(sm_m[threadIdx.x] - sm_mx[threadIdx.x & 15]);
  __syncthreads();
  if (threadIdx.x < 16) {
    float den = 0.f;
    for (int w = 0; w < W; ++w) den += sm_f[w * 16 + threadIdx.x] * sm_l[w * 16 + threadIdx.x];
    sm_den[threadIdx.x] = den;
  }
  __syncthreads();

  // Output position e = (source lane, n, v): node row 4*(lane/16)+v, dim
  // NO*(lane%16)+n; its value is sum_w f_w O_w (unnormalised) in wave order.
  const size_t tile = (size_t)head * gridDim.y + qt;       // (head, node tile)
  float* pm = a.part_ml + (tile * G + g) * 32;             // [16][2]
  float* po = a.part_o + (tile * G + g) * 16 * HD;         // [16][HD]
  for (int e = threadIdx.x; e < 64 * NO * 4; e += blockDim.x) {
    const int src = e / (NO * 4), n = (e / 4) % NO, v = e % 4;
    const int row = (src >> 4) * 4 + v;
    if (row >= rows) continue;
    const int node = row0 + row;
    float num = 0.f;
    for (int w = 0; w < W; ++w) num += sm_f[w * 16 + row] * sm_o[(w * 64 + src) * OS + n * 4 + v];
    const int dim = NO * (src & 15) + n;
    if (G == 1)
      store_act<TW>(a.o, a.o_plane, act_index<TW>(node, head * HD + dim, a.d), num / sm_den[row]);
    else
      po[row * HD + dim] = num;
  }
  if (G > 1 && threadIdx.x < 16) {
    pm[threadIdx.x * 2 + 0] = sm_mx[threadIdx.x];
    pm[threadIdx.x * 2 + 1] = sm_den[threadIdx.x];
  }
  if (G == 1) return;

  // Publish this workgroup's partial, then let the last arrival merge.  The
  // barrier completes every wave's stores; one thread's device-scope fence
  // then releases them (and, in the last workgroup, acquires the others'):
  // on this multi-XCD part a fence writes back / invalidates L2, so it is
  // issued once per workgroup, not per thread.
  __shared__ int last;
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    const int prev = atomicAdd(a.counters + tile, 1);
    last = prev == G - 1;
    if (last) __threadfence();
  }
  __syncthreads();
  if (!last) return;
  const float* pm0 = a.part_ml + tile * G * 32;
  const float* po0 = a.part_o + tile * G * 16 * HD;
  for (int e = threadIdx.x; e < 16 * HD; e += blockDim.x) {
    const int row = e / HD, dim = e % HD;
    if (row >= rows) continue;
    const int node = row0 + row;
    float mx = -1e30f;
    for (int k = 0; k < G; ++k) mx = fmaxf(mx, pm0[k * 32 + row * 2]);
    float num = 0.f, den = 0.f;
    for (int k = 0; k < G; ++k) {
      const float f = exp2f(pm0[k * 32 + row * 2] - mx);
      den += f * pm0[k * 32 + row * 2 + 1];
      num += f * po0[(size_t)k * 16 * HD + row * HD + dim];
    }
    store_act<TW>(a.o, a.o_plane, act_index<TW>(node, head * HD + dim, a.d), num / den);
  }
  if (threadIdx.x == 0) a.counters[tile] = 0;
}

template <typename TK, int HD>
constexpr size_t attn_lds() {
  return (size_t)(64 * (HD / 4 * (int)sizeof(TK) / 16) * 4 + kAttnWaves * 16 * 2 + kAttnWaves * 64 * (HD / 4 + 1) +
                  16 + kAttnWaves * 16 + 16) * 4;
}

template <typename TK, typename TW, int HD>
static hipError_t attn_attr() {
  return hipFuncSetAttribute((const void*)k_attn<TK, TW, HD>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)attn_lds<TK, HD>());
}

// Raises the LDS limit of the attention kernels (more than 64 KiB); done once
// at context creation so that no attribute call falls inside a captured step.
hipError_t init_kernel_attributes() {
  hipError_t e = attn_attr<_Float16, __bf16, 128>();
  if (e == hipSuccess) e = attn_attr<_Float16, __bf16, 64>();
  if (e == hipSuccess) e = attn_attr<float, float, 128>();
  if (e == hipSuccess) e = attn_attr<float, float, 64>();
  return e;
}

template <typename TK, typename TW, int HD>
static hipError_t attn_t(int qt, const AttnArgs& a, hipStream_t s) {
  const size_t lds = attn_lds<TK, HD>();
  TSS_LAUNCH((k_attn<TK, TW, HD>), dim3(a.n_heads, qt, a.groups), dim3(kAttnWaves * 64), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_attn(bool bf16, int head_dim, int qt, const AttnArgs& a, hipStream_t s) {
  if (bf16)
    return head_dim == 128 ? attn_t<_Float16, __bf16, 128>(qt, a, s) : attn_t<_Float16, __bf16, 64>(qt, a, s);
  return head_dim == 128 ? attn_t<float, float, 128>(qt, a, s) : attn_t<float, float, 64>(qt, a, s);
}

}  // namespace tss
