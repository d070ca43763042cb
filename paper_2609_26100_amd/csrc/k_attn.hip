// Tree-masked attention of the verify step over the paged KV cache (gfx950).
//
// For every head and node i: softmax(q_i K^T / sqrt(hd)) V over the cached
// context [0, n_kv) plus the draft nodes visible to i (i itself and its
// ancestors; their K/V were appended at slots n_kv + j by the QKV kernel).
// This is the attention half of an active block; bypassed blocks never reach
// this kernel (Domain-Aware Skip Controller, block rule).
//
// One wavefront owns (KV split, head, 16-node tile) and walks its pages:
//   * K page block [16 tokens][hd] is read with one contiguous 64-byte run per
//     lane (the whole 4 KiB block per wave), and S = K Q^T comes out of MFMA
//     with tokens on the rows and nodes on the columns.
//   * The S accumulator layout (lane: node column, 4 token rows) is exactly
//     the A-operand layout of the P V product, so probabilities never leave
//     registers.  The V block is stored [4][hd][4] so each lane's B operand for
//     all hd/16 output tiles is again one contiguous 64-byte run.
//   * Online softmax in the exp2 domain, fp32; masked keys get -inf.
//   * Operands: fp16 K/V pages, q and probabilities with fp32 accumulation
//     (v_mfma_f32_16x16x32_f16 for S, v_mfma_f32_16x16x16_f16 for P V) in the
//     bf16 mode; fp32 throughout (v_mfma_f32_16x16x4_f32) in the f32 mode.
// Splits write (max, sum, unnormalised output) partials; k_combine merges them
// in a fixed order, so results are bit-reproducible.
#include "tss_internal.h"

namespace tss {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ unsigned pack_f16x2(float lo, float hi) {
  const _Float16 a = (_Float16)lo, b = (_Float16)hi;
  return (unsigned)__builtin_bit_cast(unsigned short, a) | ((unsigned)__builtin_bit_cast(unsigned short, b) << 16);
}

// T = KV element type (_Float16 or float).
template <typename T, int HD>
__global__ __launch_bounds__(64) void k_attn(AttnArgs a) {
  constexpr int DL = HD / 4;                    // dims per lane group in Q K^T
  constexpr int NQ = DL * (int)sizeof(T) / 16;  // 16-byte K/Q chunks per lane
  constexpr int NO = HD / 16;                   // output tiles of P V
  constexpr int NV = NO * 4 * (int)sizeof(T) / 16;  // 16-byte V chunks per lane

  const int split = blockIdx.x, head = blockIdx.y, qt = blockIdx.z;
  const int lane = threadIdx.x, r16 = lane & 15, grp = lane >> 4;
  const int M = a.M, n_kv = a.n_kv;
  const int qn = qt * 16 + r16;

  // B operand of S = K Q^T: lane (node qn, group grp) holds q[qn][head*HD + grp*DL + 0..DL).
  uint4 qreg[NQ];
  {
    const float* qrow = a.q + (size_t)qn * a.d + head * HD + grp * DL;
#pragma unroll
    for (int c = 0; c < NQ; ++c) {
      if (qn < M) {
        if constexpr (sizeof(T) == 2) {
          const float4 f0 = *(const float4*)(qrow + c * 8);
          const float4 f1 = *(const float4*)(qrow + c * 8 + 4);
          qreg[c] = uint4{pack_f16x2(f0.x, f0.y), pack_f16x2(f0.z, f0.w), pack_f16x2(f1.x, f1.y),
                          pack_f16x2(f1.z, f1.w)};
        } else {
          qreg[c] = *(const uint4*)(qrow + c * 4);
        }
      } else {
        qreg[c] = uint4{0, 0, 0, 0};
      }
    }
  }
  const uint64_t anc = qn < M ? a.sp->anc[qn] : 0ull;

  const int total = n_kv + M;
  const int n_pages = (total + kPage - 1) / kPage;
  const int p0 = split * a.pages_per_split;
  const int p1 = min(p0 + a.pages_per_split, n_pages);

  float m_run = -1e30f, l_run = 0.f;
  f32x4 O[NO];
#pragma unroll
  for (int n = 0; n < NO; ++n) O[n] = f32x4{0.f, 0.f, 0.f, 0.f};

  const size_t blk_elems = 16 * (size_t)HD;
  for (int p = p0; p < p1; ++p) {
    const int phys = a.page_table[p];
    const T* kb = (const T*)a.kv_pages + (((size_t)a.layer * a.n_pages_pool + phys) * 2 * a.n_heads + head) * blk_elems;
    const T* vb = kb + (size_t)a.n_heads * blk_elems;
    uint4 kreg[NQ], vreg[NV];
    const uint4* kp = (const uint4*)(kb + r16 * HD + grp * DL);
    const uint4* vp = (const uint4*)(vb + grp * HD * 4 + r16 * NO * 4);
#pragma unroll
    for (int c = 0; c < NQ; ++c) kreg[c] = kp[c];
#pragma unroll
    for (int c = 0; c < NV; ++c) vreg[c] = vp[c];

    f32x4 S = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NQ; ++c) {
      if constexpr (sizeof(T) == 2) {
        S = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, kreg[c]),
                                                   __builtin_bit_cast(f16x8, qreg[c]), S, 0, 0, 0);
      } else {
        S = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kreg[c].x), __uint_as_float(qreg[c].x), S, 0, 0, 0);
        S = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kreg[c].y), __uint_as_float(qreg[c].y), S, 0, 0, 0);
        S = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kreg[c].z), __uint_as_float(qreg[c].z), S, 0, 0, 0);
        S = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kreg[c].w), __uint_as_float(qreg[c].w), S, 0, 0, 0);
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
        vis = j < M && ((anc >> j) & 1ull);
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

    if constexpr (sizeof(T) == 2) {
      // A = P[node r16][tokens 4*grp..+3]; B = V[tokens 4*grp..+3][dim NO*r16 + n]
      const unsigned p01 = pack_f16x2(pv[0], pv[1]), p23 = pack_f16x2(pv[2], pv[3]);
      const f16x4 A = __builtin_bit_cast(f16x4, uint2{p01, p23});
      const uint2* v2 = (const uint2*)vreg;
#pragma unroll
      for (int n = 0; n < NO; ++n)
        O[n] = __builtin_amdgcn_mfma_f32_16x16x16f16(A, __builtin_bit_cast(f16x4, v2[n]), O[n], 0, 0, 0);
    } else {
      const float* vf = (const float*)vreg;
#pragma unroll
      for (int v = 0; v < 4; ++v)
#pragma unroll
        for (int n = 0; n < NO; ++n)
          O[n] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[v], vf[n * 4 + v], O[n], 0, 0, 0);
    }
  }

  const size_t pbase = ((size_t)head * a.nsplit + split) * a.Mp;
  if (grp == 0 && qn < M) {
    a.part_ml[(pbase + qn) * 2 + 0] = m_run;
    a.part_ml[(pbase + qn) * 2 + 1] = l_run;
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int node = qt * 16 + grp * 4 + v;
    if (node < M) {
      float* dst = a.part_o + (pbase + node) * HD + NO * r16;
#pragma unroll
      for (int n = 0; n < NO; ++n) dst[n] = O[n][v];
    }
  }
}

// T = weight type of the mode (selects the activation plane format of o).
template <typename T, int HD>
__global__ __launch_bounds__(HD) void k_combine(CombineArgs a) {
  const int head = blockIdx.x, node = blockIdx.y, dim = threadIdx.x;
  const size_t base = (size_t)head * a.nsplit * a.Mp;
  float mx = -1e30f;
  for (int s = 0; s < a.nsplit; ++s) mx = fmaxf(mx, a.part_ml[(base + (size_t)s * a.Mp + node) * 2]);
  float num = 0.f, den = 0.f;
  for (int s = 0; s < a.nsplit; ++s) {
    const size_t r = base + (size_t)s * a.Mp + node;
    const float w = exp2f(a.part_ml[r * 2] - mx);
    den += w * a.part_ml[r * 2 + 1];
    num += w * a.part_o[r * HD + dim];
  }
  store_act<T>(a.o, a.o_plane, (size_t)node * a.d + head * HD + dim, num / den);
}

template <typename T, int HD>
static hipError_t attn_t(int qt, const AttnArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k_attn<T, HD>), dim3(a.nsplit, a.n_heads, qt), dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_attn(bool bf16, int head_dim, int qt, const AttnArgs& a, hipStream_t s) {
  if (bf16) return head_dim == 128 ? attn_t<_Float16, 128>(qt, a, s) : attn_t<_Float16, 64>(qt, a, s);
  return head_dim == 128 ? attn_t<float, 128>(qt, a, s) : attn_t<float, 64>(qt, a, s);
}

template <typename T, int HD>
static hipError_t combine_t(const CombineArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k_combine<T, HD>), dim3(a.n_heads, a.M), dim3(HD), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_combine(bool bf16, int head_dim, const CombineArgs& a, hipStream_t s) {
  if (bf16) return head_dim == 128 ? combine_t<__bf16, 128>(a, s) : combine_t<__bf16, 64>(a, s);
  return head_dim == 128 ? combine_t<float, 128>(a, s) : combine_t<float, 64>(a, s);
}

}  // namespace tss
