// Weight-streaming projection GEMM for the verify step on gfx950.
//
// y[m][n] = sum_k x[m][k] * W[n][k] for the few rows m of one verify step
// (the root and its drafted nodes), i.e. the Q/K/V, O, gate/up, down and
// lm_head projections of a LLaMA block (the block's attention and
// feed-forward work that the skip rule removes for bypassed layers).
//
// At a handful of rows the product is bound by streaming W from HBM, so the
// design is about bytes, not FLOPs:
//   * W is pre-packed in 1 KiB MFMA-lane-ordered tiles (tss_internal.h): every
//     wave-wide 16-byte load reads one contiguous KiB, and a workgroup streams
//     one strip of 16 (or 32) output columns over the full K.
//   * The waves of a workgroup split K; each wave keeps a ring of chunk
//     loads in flight (refilled as each chunk is consumed), runs the MFMAs,
//     and the partial sums meet in LDS in a fixed order (no atomics: results
//     are bit-reproducible).
//   * Rows are padded to 16 for the MFMA; padded rows load nothing.
//   * fp16 (the bf16-weight mode): W and the activations in fp16, one
//     v_mfma_f32_16x16x32_f16 per tile and chunk.  f32: four
//     v_mfma_f32_16x16x4_f32 per 16-byte chunk.
// Epilogues fuse the element-wise work around each projection:
//   EPI_QKV     RMSNorm row scale, rotate-half RoPE at each node's position,
//               q to the workspace, k and v into the node's paged KV slot.
//   EPI_RESID   residual add into h, then the next RMSNorm's input
//               h * gain (activation planes) and per-strip sums of h^2.
//   EPI_SWIGLU  RMSNorm row scale, silu(gate) * up.
//   EPI_LOGITS  RMSNorm row scale, fp32 logits and per-strip argmax.
#include "tss_internal.h"

namespace tss {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <typename T>
__device__ __forceinline__ f32x4 mfma_chunk(const uint4& a, const uint4& b, f32x4 c);

template <>
__device__ __forceinline__ f32x4 mfma_chunk<_Float16>(const uint4& a, const uint4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                0, 0);
}

template <>
__device__ __forceinline__ f32x4 mfma_chunk<float>(const uint4& a, const uint4& b, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  return c;
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// Weight tiles are read exactly once per step: nontemporal loads keep them
// from displacing the activations that every workgroup re-reads from L2.
__device__ __forceinline__ uint4 load_stream(const uint8_t* p) {
  typedef unsigned int u4v __attribute__((ext_vector_type(4)));
  const u4v v = __builtin_nontemporal_load((const u4v*)p);
  return uint4{v.x, v.y, v.z, v.w};
}

// Chunks each wave keeps in flight: a ring of D slots, each holding one
// chunk's weight tiles (NT x 4 VGPRs) and activation tiles (MT x S x 4
// VGPRs), sized to a VGPR budget per lane: 64 with one row tile, where more
// would cost occupancy, and with the largest accumulator sets (20+ tiles),
// where more would spill; 128 between.  The one-row-tile gate/up takes 32
// (two slots): its many workgroups then fit three to a CU, and with that many
// waves a shallower ring streams faster (7B k=5 step 3168 -> 3138 us); the
// one-row-tile lm_head likewise (three workgroups per CU: 47.7 -> 46.7 us).  The
// one-row-tile Q/K/V takes 48 (two slots of its three-tile blocks: 19.3 ->
// 19.0 us on the 7B shape) and 36 in one-tile blocks (three slots in 76
// VGPRs, so three workgroups share a CU; 48 would take 84); budgets of 96-192
// slow Q/K/V, O and down (by 0.5-1 us each), 48 slows down (19.0 -> 19.4 us)
// and 32 the whole step.  Measured on the 7B projections.
template <int MT, int NT, int S, int EPI> struct Depth {
  static constexpr int per = NT * 4 + MT * S * 4;
  static constexpr int budget = MT == 1 ? (EPI == EPI_SWIGLU || EPI == EPI_LOGITS ? 32 : (EPI == EPI_QKV ? (NT == 1 ? 36 : 48) : 64)) : (MT * NT >= 20 ? 64 : 128);
  static constexpr int raw = budget / per;
  static constexpr int v = raw < 1 ? 1 : (raw > 8 ? 8 : raw);
};

// dynamic LDS of the many-row variants: the CU's 160 KiB less room for the
// kernel's static per-row arrays; the one-row-tile and narrow variants stay
// within 64 KiB (measured faster)
constexpr size_t kGemmLdsMax = 152 * 1024;
template <int MT, int NT>
constexpr size_t gemm_lds_cap() { return (MT == 1 || (MT <= 4 && NT <= 2)) ? 65536 : kGemmLdsMax; }

// Cross-wave reduction in column passes of RC columns: the widest pass (a
// multiple of 16 dividing the block's columns) for which the 8 waves'
// partial tiles [8][ROWS][RC + pad], the summed tile yfin [ROWS][COLS], the
// residual epilogue's squares aux [ROWS][COLS] and the row scales fit the
// LDS cap, so every variant keeps 8 waves.  With several row tiles the rows
// of the partial tiles are padded by 4 floats: a wave writes rows 4 apart
// from its four 16-lane groups, which then fall on different LDS banks.
// With several row tiles the gate/up passes apply SwiGLU and store straight
// from the partial tiles (whole gate/up pairs per pass), so that block keeps
// neither yfin nor aux and its passes can be wider.
template <int MT>
constexpr int red_pad() { return MT >= 2 ? 4 : 0; }
template <int MT, int EPI>
constexpr bool fused_epi() { return EPI == EPI_SWIGLU && MT >= 2; }
template <int MT, int NT, int EPI>
constexpr size_t gemm_lds_floats(int waves, int rc) {
  return (size_t)waves * MT * 16 * (rc + red_pad<MT>()) + (fused_epi<MT, EPI>() ? 0 : 2 * MT * 16 * NT * 16) + MT * 16;
}
template <int MT, int NT, int EPI>
constexpr int red_cols() {
  for (int t = NT; t > 1; --t)
    if (NT % t == 0 && (!fused_epi<MT, EPI>() || t % 2 == 0) &&
        gemm_lds_floats<MT, NT, EPI>(8, 16 * t) * 4 <= gemm_lds_cap<MT, NT>())
      return 16 * t;
  return fused_epi<MT, EPI>() ? 32 : 16;
}
template <int MT, int NT, int EPI>
constexpr size_t gemm_lds(int waves) {
  return gemm_lds_floats<MT, NT, EPI>(waves, red_cols<MT, NT, EPI>()) * 4;
}

// Epilogue operands of the one-row-tile residual epilogue (one output item
// per thread): h and, when every row belongs to segment 0, the next norm's
// gain, requested after the wave's last weight chunk, so no weight load waits
// behind them, and in flight while the last MFMAs and the cross-wave
// reduction run.  Their addresses need no other load, and every thread loads
// (its index clamped to a valid item), so the load-count waits stay exact.
template <int EPI, int MT, int COLS>
__device__ __forceinline__ void prefetch_epilogue(const GemmArgs& a, int M, int n0, float4& pre_h, float4& pre_g) {
  if constexpr (EPI == EPI_RESID && MT == 1) {
    const int e4 = min((int)threadIdx.x, M * COLS / 4 - 1);
    const int row = e4 / (COLS / 4), col = (e4 % (COLS / 4)) * 4;
    pre_h = *(const float4*)(a.h + (size_t)row * a.N + n0 + col);
    pre_g = *(const float4*)(a.g_next[0] + n0 + col);
  }
}

// Row r's segment runs this block: bit r of the two row_on words, read as
// uniform values (scalar loads) with the bit selected per lane.  (Indexing
// the argument block per lane instead makes a vector load from it, whose wait
// sits in every epilogue iteration.)
static_assert(kMaxRows == 128, "two words of row bits");
struct RowBits {
  uint64_t w0, w1;
  __device__ __forceinline__ explicit RowBits(const GemmArgs& a) : w0(a.row_on[0]), w1(a.row_on[1]) {}
  __device__ __forceinline__ bool on(int r) const { return ((r < 64 ? w0 : w1) >> (r & 63)) & 1ull; }
};

// The workgroup's projection: its strip (blockIdx.x, with a K split
// blockIdx.x / ksplit); for gate/up its NT / 2 pairs from strip * NT / 2 on,
// or from pair0 on in launches of two block widths (GIVEN).
template <typename T, int MT, int NT, int EPI, bool GIVEN = false>
__device__ __forceinline__ void gemm_body(GemmArgs a, int pair0 = 0) {
  constexpr int KC = 64 / sizeof(T);   // K elements per 1 KiB tile
  constexpr int KL = KC / 4;           // K elements per lane per tile
  constexpr int S = Mode<T>::planes;
  // ring depths were tuned with 16-bit activations in two planes; the one
  // fp16 plane keeps the same depths (its slots need half the activation
  // registers)
  constexpr int D = Depth<MT, NT, sizeof(T) == 2 ? 2 : S, EPI>::v;
  using KV = typename Mode<T>::KV;
  constexpr int ROWS = MT * 16;
  constexpr int COLS = NT * 16;
  extern __shared__ float smem[];

  const int waves = blockDim.x >> 6;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r16 = lane & 15, grp = lane >> 4;
  const int M = a.M, K = a.K, nkc = a.nkc;
  // strip and, with a K split, this workgroup's chunks [c_lo, c_hi) of K
  // (only the residual projections with 2+ row tiles split K: every other
  // instantiation compiles with ks = 1)
  constexpr bool SPLIT = EPI == EPI_RESID && MT >= 2;
  const int ks = SPLIT ? a.ksplit : 1;
  const int strip = SPLIT ? (int)blockIdx.x / ks : (int)blockIdx.x;
  const int split = SPLIT ? (int)blockIdx.x - strip * ks : 0;
  const int c_lo = SPLIT ? split * nkc / ks : 0, c_hi = SPLIT ? (split + 1) * nkc / ks : nkc;
  if constexpr (!GIVEN) pair0 = strip * (NT / 2);
  // weight tile nt of this strip, chunk c, at wb[nt] + c * wstep: plain
  // matrices store a 16-row tile's chunks consecutively; gate and up tiles of
  // one pair alternate chunk by chunk
  const uint8_t* wb[NT];
  size_t wstep;
  if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      wb[nt] = a.w + (((size_t)(pair0 + nt / 2) * nkc * 2) + (nt & 1)) * kTileBytes + lane * 16;
    wstep = 2 * kTileBytes;
  } else {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) wb[nt] = a.w + (size_t)(strip * NT + nt) * nkc * kTileBytes + lane * 16;
    wstep = kTileBytes;
  }
  const T* x = (const T*)a.x;

  f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Per-row data the epilogue needs (sequence, KV slot, rotary position),
  // staged before the weight stream so its latency hides behind it.
  __shared__ int s_seq[EPI == EPI_QKV || EPI == EPI_RESID ? kMaxRows : 1];
  __shared__ int s_slot[EPI == EPI_QKV ? kMaxRows : 1];
  __shared__ int s_pos[EPI == EPI_QKV ? kMaxRows : 1];
  __shared__ int s_page[EPI == EPI_QKV ? kMaxRows : 1];                // KV page of the row's slot
  __shared__ int2 s_col[EPI == EPI_QKV ? COLS : 1];  // per column: section | head << 2, dim | rotary index << 16
  __shared__ const float* s_gain[EPI == EPI_RESID ? kMaxRows : 1];    // next-norm gain of the row's segment
  if constexpr (EPI == EPI_QKV || EPI == EPI_RESID) {
    for (int r = threadIdx.x; r < M; r += blockDim.x) {
      const int sq = a.n_seqs == 1 ? 0 : a.sp->row_seq[r];
      s_seq[r] = sq;
      if constexpr (EPI == EPI_QKV) {
        const int nkv = a.sp->seq_nkv[sq];
        // local node j of segment sq sits at slot n_kv + seg_slot0 + j
        s_slot[r] = nkv + a.sp->seg_slot0[sq] + r - a.sp->seq_row0[sq];
        s_pos[r] = nkv + a.sp->depth[r];
      }
    }
  }

  // The RMSNorm partial sums of this wave's row are loaded before the weight
  // stream (when every row has its own wave), so their latency hides behind it.
  constexpr int SSV = 8;  // parts per lane: up to 512 parts per row
  const bool ss_early = a.ss_in && M <= waves;
  float ssv[SSV];
#pragma unroll
  for (int i = 0; i < SSV; ++i) {
    const int p = lane + 64 * i;
    ssv[i] = (ss_early && wave < M && p < a.ss_nparts) ? a.ss_in[(size_t)wave * a.ss_stride + p] : 0.f;
  }

  // Wave w takes chunks w, w + waves, w + 2 waves, ... (adjacent waves read
  // adjacent KiB).  Software pipeline: a ring of D slots, each refilled with
  // the chunk D steps ahead as soon as it is consumed, so D chunks stay in
  // flight through the K loop.  Activation loads are issued with their
  // chunk's weight loads (loads complete in order, so waiting on one slot
  // never waits on a later chunk).  The loads carry no conditions (the
  // counter-based waits stay exact): padded rows re-read row M-1 (their
  // products land in output rows that are never stored) and the main loop
  // only runs while every refill is in range; the last chunks are finished
  // by a short tail.
  const int nkc_s = c_hi - c_lo;
  const int n_my = wave < nkc_s ? (nkc_s - wave + waves - 1) / waves : 0;
  uint4 wv[D][NT];
  uint4 xv[D][MT][S];
  // Activation tiles through a buffer resource: a padded row (>= M) gets an
  // offset past the buffer's end, which the hardware answers with zeros
  // without touching memory (no branch, so the load-count waits stay exact).
  const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
      (void*)x, (short)0, (int)((size_t)S * (a.x_plane > 0 ? a.x_plane : (size_t)a.Mp * K) * sizeof(T)), 0x00020000);
  constexpr int kPastEnd = 1 << 30;
  int xoff[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
    xoff[mt] = mt * 16 + r16 < M ? (mt * nkc * 64 + lane) * 16 : kPastEnd;
  const int plane_bytes = (int)(a.x_plane * sizeof(T));
  auto issue = [&](uint4 (&w)[NT], uint4 (&xs)[MT][S], int i) {
    const int c = c_lo + wave + i * waves;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) w[nt] = load_stream(wb[nt] + (size_t)c * wstep);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int p = 0; p < S; ++p) {
        typedef unsigned int u4v __attribute__((ext_vector_type(4)));
        const u4v v = __builtin_amdgcn_raw_buffer_load_b128(xres, xoff[mt] + c * kTileBytes + p * plane_bytes, 0, 0);
        xs[mt][p] = uint4{v.x, v.y, v.z, v.w};
      }
  };
  auto compute = [&](uint4 (&w)[NT], uint4 (&xs)[MT][S]) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int p = 0; p < S; ++p) acc[mt][nt] = mfma_chunk<T>(xs[mt][p], w[nt], acc[mt][nt]);
  };
  // epilogue operands prefetched after the weight stream (prefetch_epilogue;
  // a wave without chunks loads them in the epilogue)
  constexpr bool PRE_RESID = EPI == EPI_RESID && MT == 1;
  float4 pre_h = make_float4(0.f, 0.f, 0.f, 0.f), pre_g = make_float4(0.f, 0.f, 0.f, 0.f);
  if (n_my > 0) {
#pragma unroll
    for (int j = 0; j < D; ++j) issue(wv[j], xv[j], min(j, n_my - 1));
    int i0 = 0;
    for (; i0 + 2 * D <= n_my; i0 += D) {
#pragma unroll
      for (int j = 0; j < D; ++j) {
        compute(wv[j], xv[j]);
        issue(wv[j], xv[j], i0 + j + D);
      }
    }
    // tail: fewer than 2 D chunks left, the first D of them already in the ring
#pragma unroll
    for (int j = 0; j < D; ++j) {
      if (i0 + j < n_my) {
        compute(wv[j], xv[j]);
        if (i0 + j + D < n_my) issue(wv[j], xv[j], i0 + j + D);
      }
    }
    if constexpr (PRE_RESID) prefetch_epilogue<EPI, MT, COLS>(a, M, strip * COLS, pre_h, pre_g);
#pragma unroll
    for (int j = 0; j < D; ++j)
      if (i0 + D + j < n_my) compute(wv[j], xv[j]);
  }

  // Per-row lookups of the epilogue that depend on the prologue's row data
  // (each thread reads the rows it wrote there), requested now so they land
  // while the waves' partial tiles are reduced; the reduction's barriers
  // publish them.
  const RowBits rows(a);
  if constexpr (EPI == EPI_QKV) {
    for (int r = threadIdx.x; r < M; r += blockDim.x) {
      const int lp = s_slot[r] >> 4;
      if (rows.on(r)) s_page[r] = lp < a.n_arg_pages ? a.pages[lp] : a.page_table[a.pt_off[s_seq[r]] + lp];
    }
    // the strip's columns: section (q, k, v), head, the head dimension the
    // packing put there and its rotary index (divisions once per column)
    const int d16 = a.d >> 4, hd16 = a.head_dim >> 4;
    for (int col = threadIdx.x; col < COLS; col += blockDim.x) {
      const int n = strip * COLS + col;
      const int tile = n >> 4, c = n & 15;
      const int sec = tile / d16, ts = tile % d16;
      const int head = ts / hd16, t = ts % hd16;
      const int dim = c < 8 ? 8 * t + c : (a.head_dim >> 1) + 8 * t + (c - 8);
      s_col[col] = make_int2(sec | head << 2, dim | (8 * t + (c & 7)) << 16);
    }
  }
  if constexpr (EPI == EPI_RESID) {
    if (a.n_seqs > 1)
      for (int r = threadIdx.x; r < M; r += blockDim.x) s_gain[r] = a.g_next[s_seq[r]];
  }

  // LDS: red[waves][ROWS][RCP] | yfin[ROWS][COLS] | aux[ROWS][COLS] | rscale[ROWS]
  // (gate/up with several row tiles: red | rscale).  The waves' partial tiles
  // meet in red one pass of RC columns at a time (rows RCP floats apart);
  // their sum lands in yfin, the residual epilogue's squares in aux.
  constexpr bool FUSED = fused_epi<MT, EPI>();
  constexpr int RC = red_cols<MT, NT, EPI>();
  constexpr int RCP = RC + red_pad<MT>();
  float* red = smem;
  float* yfin = red + waves * ROWS * RCP;
  float* aux = yfin + (FUSED ? 0 : ROWS * COLS);
  float* rscale = aux + (FUSED ? 0 : ROWS * COLS);

  // RMSNorm row scale from the producer's partial sums (fixed order, so every
  // workgroup derives the same value): here when each row has its own wave
  // (loaded before the weight stream), otherwise below.
  if (ss_early && wave < M) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < SSV; ++i) s += ssv[i];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
    if (lane == 0) rscale[wave] = rsqrtf(s / (float)a.norm_dim + a.eps);
  }

  // With several row tiles, the row scales come from eight threads per row,
  // each summing a contiguous eighth of the row's partial sums, then three
  // exchanges (a fixed order), in rounds of 64 rows.  Where the row splits
  // into eighths of whole 16-byte groups, the groups are requested before the
  // waves' partial tiles go to LDS, so their latency overlaps those writes;
  // other row widths (small models) load and add their parts one by one,
  // the parts past the row counting as zero.  Either way the scales are in
  // LDS before the first pass sums.
  constexpr int kSsq = 16;  // groups of four parts per thread: up to 512 parts per row
  const bool ss_vec = MT >= 2 && a.ss_in;
  const int nq4 = (a.ss_nparts + 31) / 32;
  const bool ss_wide = a.ss_nparts % 32 == 0 && a.ss_stride % 4 == 0;  // 16-byte loads
  float4 ssq[MT >= 2 ? kSsq : 1];
  auto ss_load = [&](int r0) {
    if constexpr (MT >= 2) {
      const int row = min(r0 + ((int)threadIdx.x >> 3), M - 1);  // clamped: every thread loads
      const float* src = a.ss_in + (size_t)row * a.ss_stride + (threadIdx.x & 7) * nq4 * 4;
      if (ss_wide) {
#pragma unroll
        for (int i = 0; i < kSsq; ++i)
          if (i < nq4) ssq[i] = *(const float4*)(src + 4 * i);
      }
    }
  };
  auto ss_finish = [&](int r0) {
    if constexpr (MT >= 2) {
      float t = 0.f;
      if (ss_wide) {
#pragma unroll
        for (int i = 0; i < kSsq; ++i)
          if (i < nq4) t += (ssq[i].x + ssq[i].y) + (ssq[i].z + ssq[i].w);
      } else {
        const int row = min(r0 + ((int)threadIdx.x >> 3), M - 1);
        const int p0 = (threadIdx.x & 7) * nq4 * 4;
        const float* src = a.ss_in + (size_t)row * a.ss_stride;
        for (int q = p0; q < p0 + nq4 * 4; ++q) t += q < a.ss_nparts ? src[q] : 0.f;
      }
      t += __shfl_xor(t, 1);
      t += __shfl_xor(t, 2);
      t += __shfl_xor(t, 4);
      const int row = r0 + ((int)threadIdx.x >> 3);
      if ((threadIdx.x & 7) == 0 && row < M) rscale[row] = rsqrtf(t / (float)a.norm_dim + a.eps);
    }
  };
  if (ss_vec) ss_load(0);

  // When the row scale is known before the sums (loaded early or just above,
  // or no norm), it is applied as they are written (the same product as
  // applying it afterwards), which saves a pass over the block and a
  // barrier.  The residual projections (no norm, possibly K-split) always
  // fold.
  const bool fold = ss_early || !a.ss_in || ss_vec;

  // MFMA result layout: lane holds column r16, rows 4*grp + v.
#pragma unroll
  for (int c0 = 0; c0 < COLS; c0 += RC) {
    if (c0 > 0) __syncthreads();  // the previous pass has read red
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = c0 / 16; nt < (c0 + RC) / 16; ++nt)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          red[(wave * ROWS + mt * 16 + grp * 4 + v) * RCP + nt * 16 - c0 + r16] = acc[mt][nt][v];
    if (c0 == 0 && ss_vec) {
      ss_finish(0);
      for (int r0 = (int)blockDim.x / 8; r0 < M; r0 += (int)blockDim.x / 8) {
        ss_load(r0);
        ss_finish(r0);
      }
    }
    __syncthreads();
    if constexpr (FUSED) {
      // gate/up: four adjacent outputs of a pair per thread, gate and up
      // summed in wave order, scaled, silu(gate) * up, one vector store per
      // plane (the same operations as summing into yfin first)
      constexpr int PP = RC / 32;  // gate/up pairs per pass
      const int F = a.N >> 1;
      for (int it = threadIdx.x; it < M * PP * 4; it += blockDim.x) {
        const int row = it / (PP * 4), jp = (it >> 2) % PP, c = (it & 3) * 4;
        const float* rg = red + row * RCP + jp * 32 + c;
        float4 g = make_float4(0.f, 0.f, 0.f, 0.f), u = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int w = 0; w < waves; ++w) {
          const float4 gw = *(const float4*)(rg + w * ROWS * RCP);
          const float4 uw = *(const float4*)(rg + w * ROWS * RCP + 16);
          g.x += gw.x; g.y += gw.y; g.z += gw.z; g.w += gw.w;
          u.x += uw.x; u.y += uw.y; u.z += uw.z; u.w += uw.w;
        }
        if (a.ss_in) {
          const float r = rscale[row];
          g = make_float4(g.x * r, g.y * r, g.z * r, g.w * r);
          u = make_float4(u.x * r, u.y * r, u.z * r, u.w * r);
        }
        store_act4<T>(a.act, a.act_plane, act_index<T>(row, (pair0 + c0 / 32 + jp) * 16 + c, F),
                      make_float4(silu(g.x) * u.x, silu(g.y) * u.y, silu(g.z) * u.z, silu(g.w) * u.w));
      }
    } else {
      for (int e = threadIdx.x; e < M * RC; e += blockDim.x) {
        const int row = e / RC, col = e % RC;
        float s = 0.f;
        for (int w = 0; w < waves; ++w) s += red[(w * ROWS + row) * RCP + col];
        yfin[row * COLS + c0 + col] = fold && a.ss_in ? s * rscale[row] : s;
      }
    }
  }

  bool split_done = false;  // the K-split merge ran the residual epilogue's element-wise part
  if (SPLIT && ks > 1) {
    // K split: publish this workgroup's sums (agent-scope stores: visible to
    // every XCD once acknowledged), count the arrival, and let the last
    // workgroup of the strip add the ks partial products in split order
    __shared__ int s_last;
    __syncthreads();  // yfin complete
    typedef float f4v __attribute__((ext_vector_type(4)));
    const size_t slot_floats = (size_t)a.Mp * COLS;
    const __amdgpu_buffer_rsrc_t pres = __builtin_amdgcn_make_buffer_rsrc(
        a.kpart, (short)0, (int)(gridDim.x * slot_floats * sizeof(float)), 0x00020000);
    constexpr int kScopeAgent = 16;  // cache-policy operand: sc1 (agent scope)
    for (int e4 = threadIdx.x; e4 < M * COLS / 4; e4 += blockDim.x)
      __builtin_amdgcn_raw_buffer_store_b128(*(const f4v*)(yfin + 4 * e4), pres,
                                             (int)((blockIdx.x * slot_floats + 4 * e4) * sizeof(float)), 0,
                                             kScopeAgent);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0)
      s_last = __hip_atomic_fetch_add(a.kcount + strip, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == ks - 1;
    __syncthreads();
    if (!s_last) return;
    // The last arrival adds the partial tiles and runs the residual
    // epilogue's element-wise part on the sums directly, two elements per
    // thread at a time, with all their requests (the other splits' partial
    // tiles, h, the next norm's gain) issued together.
    const int N = a.N, n4 = M * COLS / 4;
    for (int b0 = threadIdx.x; b0 < n4; b0 += 2 * (int)blockDim.x) {
      f4v v[2][kMaxKSplit];
      float4 h0[2], gn[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int e4 = min(b0 + u * (int)blockDim.x, n4 - 1);  // clamped: every thread loads
        const int row = e4 / (COLS / 4), col = (e4 % (COLS / 4)) * 4;
#pragma unroll
        for (int k = 0; k < kMaxKSplit; ++k)
          if (k < ks && k != split)
            v[u][k] = __builtin_amdgcn_raw_buffer_load_b128(
                pres, (int)(((size_t)(strip * ks + k) * slot_floats + 4 * e4) * sizeof(float)), 0, kScopeAgent);
        h0[u] = *(const float4*)(a.h + (size_t)row * N + strip * COLS + col);
        gn[u] = *(const float4*)((a.n_seqs == 1 ? a.g_next[0] : s_gain[row]) + strip * COLS + col);
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int e4 = b0 + u * (int)blockDim.x;
        if (e4 >= n4) break;
        const int row = e4 / (COLS / 4), col = (e4 % (COLS / 4)) * 4;
        const f4v own = *(const f4v*)(yfin + 4 * e4);
        f4v t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < kMaxKSplit; ++k)
          if (k < ks) t += k == split ? own : v[u][k];
        // rows whose sequence skips this block keep h, their next-norm input
        // and their partial sums untouched
        if (!rows.on(row)) continue;
        const float4 hn = make_float4(h0[u].x + t.x, h0[u].y + t.y, h0[u].z + t.z, h0[u].w + t.w);
        *(float4*)(a.h + (size_t)row * N + strip * COLS + col) = hn;
        store_act4<T>(a.xn, a.xn_plane, act_index<T>(row, strip * COLS + col, N),
                      make_float4(hn.x * gn[u].x, hn.y * gn[u].y, hn.z * gn[u].z, hn.w * gn[u].w));
        *(float4*)(aux + row * COLS + col) = make_float4(hn.x * hn.x, hn.y * hn.y, hn.z * hn.z, hn.w * hn.w);
      }
    }
    if (threadIdx.x == 0) a.kcount[strip] = 0;
    split_done = true;
  }

  if (!fold) {
    // rows in groups of 4 per wave, every load of a group issued together
    // (indices clamped, out-of-range parts weighted 0)
    for (int m0 = wave; m0 < M; m0 += 4 * waves) {
      float sum[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = min(m0 + r * waves, M - 1);
        float v[SSV];
#pragma unroll
        for (int i = 0; i < SSV; ++i) v[i] = a.ss_in[(size_t)m * a.ss_stride + min(lane + 64 * i, a.ss_nparts - 1)];
        float t = 0.f;
#pragma unroll
        for (int i = 0; i < SSV; ++i) t += lane + 64 * i < a.ss_nparts ? v[i] : 0.f;
        sum[r] = t;
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float t = sum[r];
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) t += __shfl_xor(t, off);
        const int m = m0 + r * waves;
        if (lane == 0 && m < M) rscale[m] = rsqrtf(t / (float)a.norm_dim + a.eps);
      }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < M * COLS; e += blockDim.x) yfin[e] *= rscale[e / COLS];
  }
  if constexpr (!FUSED) __syncthreads();

  const int n0 = strip * COLS;
  if constexpr (EPI == EPI_QKV) {
    const int HD = a.head_dim, d = a.d;
    // Elements in batches of QB per thread (what the launch gives a thread
    // with 8 waves, at most 8): the batch's rotary coefficients are requested
    // together before any of its stores, so they cost one round trip.
    constexpr int QB = (ROWS * COLS + 511) / 512 > 8 ? 8 : (ROWS * COLS + 511) / 512;
    for (int e0 = threadIdx.x; e0 < M * COLS; e0 += QB * (int)blockDim.x) {
      float2 cs[QB];
      int sec[QB], head[QB], dim[QB];
#pragma unroll
      for (int j = 0; j < QB; ++j) {
        const int e = e0 + j * (int)blockDim.x;
        if (e < M * COLS) {
          const int row = e / COLS;
          const int2 ci = s_col[e % COLS];
          sec[j] = ci.x & 3;
          head[j] = ci.x >> 2;
          dim[j] = ci.y & 0xffff;
          // every column has a rotary index (< hd / 2), so the request is in
          // bounds even where the value goes unused (v)
          cs[j] = a.rope[(size_t)s_pos[row] * (HD >> 1) + (ci.y >> 16)];
        }
      }
#pragma unroll
      for (int j = 0; j < QB; ++j) {
        const int e = e0 + j * (int)blockDim.x;
        if (e >= M * COLS) break;
        const int row = e / COLS, col = e % COLS, c = col & 15;
        float val = yfin[row * COLS + col];
        if (sec[j] < 2) {
          const float partner = yfin[row * COLS + (col ^ 8)];
          val = c < 8 ? val * cs[j].x - partner * cs[j].y : val * cs[j].x + partner * cs[j].y;
        }
        if (sec[j] == 0) {
          a.q[(size_t)row * d + head[j] * HD + dim[j]] = val;
        } else if (rows.on(row)) {
          const int tin = s_slot[row] & 15;
          KV* blk = (KV*)a.kv_pages +
                    ((((size_t)a.layer * a.n_pages_pool + s_page[row]) * 2 + (sec[j] - 1)) * a.n_heads + head[j]) *
                        (16 * (size_t)HD);
          if (sec[j] == 1)
            blk[tin * HD + dim[j]] = (KV)val;
          else
            blk[(tin >> 2) * HD * 4 + dim[j] * 4 + (tin & 3)] = (KV)val;
        }
      }
    }
  } else if constexpr (EPI == EPI_RESID) {
    // rows whose sequence skips this block keep h, their next-norm input and
    // their partial sums untouched
    // four adjacent columns per thread: vector loads and stores of h, the
    // gain and the next-norm input (adjacent in each activation plane)
    const int N = a.N;
    for (int e4 = threadIdx.x; e4 < (split_done ? 0 : M * COLS / 4); e4 += blockDim.x) {
      const int row = e4 / (COLS / 4), col = (e4 % (COLS / 4)) * 4;
      if (!rows.on(row)) continue;
      const size_t idx = (size_t)row * N + n0 + col;
      // one pass (always with one row tile): the operands prefetched for e4
      const bool pre = PRE_RESID && M * COLS / 4 <= (int)blockDim.x && n_my > 0;
      float4 h0, gn;
      if (pre)
        h0 = pre_h;
      else
        h0 = *(const float4*)(a.h + idx);
      const float* y = yfin + row * COLS + col;
      const float4 hn = make_float4(h0.x + y[0], h0.y + y[1], h0.z + y[2], h0.w + y[3]);
      *(float4*)(a.h + idx) = hn;
      if (pre && a.n_seqs == 1)
        gn = pre_g;
      else
        gn = *(const float4*)((a.n_seqs == 1 ? a.g_next[0] : s_gain[row]) + n0 + col);
      store_act4<T>(a.xn, a.xn_plane, act_index<T>(row, n0 + col, N),
                    make_float4(hn.x * gn.x, hn.y * gn.y, hn.z * gn.z, hn.w * gn.w));
      *(float4*)(aux + row * COLS + col) = make_float4(hn.x * hn.x, hn.y * hn.y, hn.z * hn.z, hn.w * hn.w);
    }
    __syncthreads();
    // one partial sum of h^2 per 16 columns (the format every norm reads)
    for (int e = threadIdx.x; e < M * NT; e += blockDim.x) {
      const int row = e / NT, j = e % NT;
      if (!rows.on(row)) continue;
      float s = 0.f;
      for (int col = j * 16; col < j * 16 + 16; ++col) s += aux[row * COLS + col];
      a.ss_out[(size_t)row * a.ss_stride + strip * NT + j] = s;
    }
  } else if constexpr (EPI == EPI_SWIGLU && !FUSED) {
    static_assert(NT % 2 == 0, "gate and up tiles pair up");
    const int F = a.N >> 1;
    constexpr int PAIRS = NT / 2;
    // four adjacent outputs per thread, one vector store per plane
    for (int e4 = threadIdx.x; e4 < M * 4 * PAIRS; e4 += blockDim.x) {
      const int row = e4 / (4 * PAIRS), j = (e4 / 4) % PAIRS, c = (e4 & 3) * 4;
      const float* g = yfin + row * COLS + j * 32 + c;
      const float* u = g + 16;
      store_act4<T>(a.act, a.act_plane, act_index<T>(row, (pair0 + j) * 16 + c, F),
                    make_float4(silu(g[0]) * u[0], silu(g[1]) * u[1], silu(g[2]) * u[2], silu(g[3]) * u[3]));
    }
  } else if constexpr (EPI == EPI_LOGITS) {
    const int N = a.N;
    for (int e = threadIdx.x; e < M * COLS; e += blockDim.x) {
      const int row = e / COLS, col = e % COLS;
      a.logits[(size_t)row * N + n0 + col] = yfin[row * COLS + col];
    }
    // one (max, argmax) per 16 columns, lowest column on ties; NaN counts as
    // the largest value (first NaN wins), as in numpy's argmax
    for (int e = threadIdx.x; e < M * NT; e += blockDim.x) {
      const int row = e / NT, j = e % NT;
      float bv = yfin[row * COLS + j * 16];
      int bi = j * 16;
      for (int col = j * 16 + 1; col < j * 16 + 16; ++col) {
        const float v = yfin[row * COLS + col];
        if (__builtin_isnan(v) ? !__builtin_isnan(bv) : v > bv) { bv = v; bi = col; }
      }
      a.am_val[(size_t)row * a.am_stride + strip * NT + j] = bv;
      a.am_idx[(size_t)row * a.am_stride + strip * NT + j] = n0 + bi;
    }
  }
}


template <typename T, int MT, int NT, int EPI>
__global__ __launch_bounds__(512) void k_gemm(GemmArgs a) {
  gemm_body<T, MT, NT, EPI>(a);
}

// Gate/up in exactly one round of 256 workgroups where the pairs do not
// divide into equal blocks that fill it: workgroups [0, wide_wgs) take
// NT / 2 pairs, the rest NT / 2 - 1 (7B with 2-4 row tiles: 176 x 3 + 80 x 2
// = 688 pairs, instead of 172 blocks of 4 pairs that leave 84 CUs idle
// while each busy CU streams 1.5 MiB; 13B with 5 row tiles: 96 x 4 + 160 x 3
// = 864 pairs, instead of 432 blocks of 2 in two rounds).
template <typename T, int MT, int NT>
__global__ __launch_bounds__(512) void k_gemm_gu2(GemmArgs a) {
  const int b = blockIdx.x;
  if (b < a.wide_wgs)
    gemm_body<T, MT, NT, EPI_SWIGLU, true>(a, b * (NT / 2));
  else
    gemm_body<T, MT, NT - 2, EPI_SWIGLU, true>(a, a.wide_wgs * (NT / 2) + (b - a.wide_wgs) * (NT / 2 - 1));
}

template <typename T, int MT, int NT, int EPI>
static hipError_t gemm_attr() {
  return hipFuncSetAttribute((const void*)k_gemm<T, MT, NT, EPI>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)kGemmLdsMax);
}

template <typename T, int MT, int NT>
static hipError_t gemm_attr_mt() {
  hipError_t e = gemm_attr<T, MT, NT, EPI_QKV>();
  if (e == hipSuccess) e = gemm_attr<T, MT, NT, EPI_RESID>();
  if (e == hipSuccess) e = gemm_attr<T, MT, NT < 2 ? 2 : NT, EPI_SWIGLU>();
  if (e == hipSuccess) e = gemm_attr<T, MT, NT, EPI_LOGITS>();
  return e;
}

// Lets the many-row variants use more than 64 KiB of LDS for the cross-wave
// reduction (called once at context creation).
template <typename T, int MT>
static hipError_t gemm_attr_rows() {
  hipError_t e = gemm_attr_mt<T, MT, 1>();
  if (e == hipSuccess) e = gemm_attr_mt<T, MT, 2>();
  if (e == hipSuccess) e = gemm_attr_mt<T, MT, 4>();
  if (e == hipSuccess) e = gemm_attr<T, MT, 3, EPI_QKV>();  // three-tile blocks: Q/K/V only
  if constexpr (MT >= 2 && MT <= 4)  // eight-tile gate/up blocks (four pairs)
    if (e == hipSuccess) e = gemm_attr<T, MT, 8, EPI_SWIGLU>();
  if constexpr (MT >= 2 && MT <= 4)  // eight-tile lm_head blocks
    if (e == hipSuccess) e = gemm_attr<T, MT, 8, EPI_LOGITS>();
  if constexpr (MT >= 2 && MT <= 4)  // gate/up blocks of three and two pairs
    if (e == hipSuccess)
      e = hipFuncSetAttribute((const void*)k_gemm_gu2<T, MT, 6>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)kGemmLdsMax);
  if constexpr (MT == 5)  // gate/up blocks of four and three pairs
    if (e == hipSuccess)
      e = hipFuncSetAttribute((const void*)k_gemm_gu2<T, MT, 8>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)kGemmLdsMax);
  if constexpr (MT >= 2 && MT <= 4)  // six-tile Q/K/V blocks
    if (e == hipSuccess) e = gemm_attr<T, MT, 6, EPI_QKV>();
  if constexpr (MT >= 2 && MT <= 3)  // ten-tile gate/up blocks (five pairs)
    if (e == hipSuccess) e = gemm_attr<T, MT, 10, EPI_SWIGLU>();
  return e;
}

hipError_t init_gemm_attributes() {
  hipError_t e = gemm_attr_rows<_Float16, 1>();
  if (e == hipSuccess) e = gemm_attr_rows<_Float16, 2>();
  if (e == hipSuccess) e = gemm_attr_rows<_Float16, 3>();
  if (e == hipSuccess) e = gemm_attr_rows<_Float16, 4>();
  if (e == hipSuccess) e = gemm_attr_rows<_Float16, 5>();
  if (e == hipSuccess) e = gemm_attr_rows<_Float16, 6>();
  if (e == hipSuccess) e = gemm_attr_rows<_Float16, 7>();
  if (e == hipSuccess) e = gemm_attr_rows<_Float16, 8>();
  if (e == hipSuccess) e = gemm_attr_rows<float, 1>();
  if (e == hipSuccess) e = gemm_attr_rows<float, 2>();
  if (e == hipSuccess) e = gemm_attr_rows<float, 3>();
  if (e == hipSuccess) e = gemm_attr_rows<float, 4>();
  return e;
}

template <typename T, int MT, int NT, int EPI>
static hipError_t launch_v(const GemmArgs& a, hipStream_t s) {
  // 8 waves (measured best across the 7B shapes) unless K is short, capped by
  // LDS: up to 64 rows the cross-wave reduction stays within 64 KiB
  // (4-tile blocks and more than 4 row tiles may use most of the CU's LDS)
  const size_t cap = gemm_lds_cap<MT, NT>();
  const int nkc_min = a.nkc / a.ksplit;  // chunks of the smallest K split
  int waves = nkc_min < 8 ? nkc_min : 8;
  while (waves > 1 && gemm_lds<MT, NT, EPI>(waves) > cap) waves >>= 1;
  const size_t lds = gemm_lds<MT, NT, EPI>(waves);
  dim3 grid(a.N / (16 * NT) * a.ksplit), block(waves * 64);
  TSS_LAUNCH((k_gemm<T, MT, NT, EPI>), grid, block, lds, s, a);
  return hipGetLastError();
}

template <typename T, int MT, int NT>
static hipError_t launch_gu2(const GemmArgs& a, hipStream_t s) {
  const int nkc_min = a.nkc;
  int waves = nkc_min < 8 ? nkc_min : 8;
  auto lds_of = [](int w) {
    const size_t lw = gemm_lds<MT, NT, EPI_SWIGLU>(w), ln = gemm_lds<MT, NT - 2, EPI_SWIGLU>(w);
    return lw > ln ? lw : ln;
  };
  while (waves > 1 && lds_of(waves) > gemm_lds_cap<MT, NT>()) waves >>= 1;
  TSS_LAUNCH((k_gemm_gu2<T, MT, NT>), dim3(kGemmRound), dim3(waves * 64), lds_of(waves), s, a);
  return hipGetLastError();
}

template <typename T, int MT, int NT>
static hipError_t launch_mt(int epi, const GemmArgs& a, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_v<T, MT, NT, EPI_QKV>(a, s);
    case EPI_RESID: return launch_v<T, MT, NT, EPI_RESID>(a, s);
    case EPI_SWIGLU: return launch_v<T, MT, NT < 2 ? 2 : NT, EPI_SWIGLU>(a, s);
    default: return launch_v<T, MT, NT, EPI_LOGITS>(a, s);
  }
}

// mt = 16-row tiles of the step's rows (up to 8 in the bf16 mode, 4 in the
// f32 mode); nt = 16-column tiles per workgroup (gemm_tiles).
template <typename T, int MT>
static hipError_t launch_rows(int epi, int nt, const GemmArgs& a, hipStream_t s) {
  switch (nt) {
    case 1: return launch_mt<T, MT, 1>(epi, a, s);
    case 2: return launch_mt<T, MT, 2>(epi, a, s);
    case 4: return launch_mt<T, MT, 4>(epi, a, s);
    case 3: return epi == EPI_QKV ? launch_v<T, MT, 3, EPI_QKV>(a, s) : hipErrorInvalidValue;
    case 8:
      if constexpr (MT >= 2 && MT <= 4)
        if (epi == EPI_LOGITS) return launch_v<T, MT, 8, EPI_LOGITS>(a, s);
      if constexpr (MT >= 2 && MT <= 4) return epi == EPI_SWIGLU ? launch_v<T, MT, 8, EPI_SWIGLU>(a, s) : hipErrorInvalidValue;
      if constexpr (MT == 5)
        if (epi == EPI_SWIGLU && a.wide_wgs > 0) return launch_gu2<T, MT, 8>(a, s);
      return hipErrorInvalidValue;
    case 6:
      if constexpr (MT >= 2 && MT <= 4) {
        if (epi == EPI_QKV) return launch_v<T, MT, 6, EPI_QKV>(a, s);
        if (epi == EPI_SWIGLU && a.wide_wgs > 0) return launch_gu2<T, MT, 6>(a, s);
      }
      return hipErrorInvalidValue;
    case 10:
      if constexpr (MT >= 2 && MT <= 3) return epi == EPI_SWIGLU ? launch_v<T, MT, 10, EPI_SWIGLU>(a, s) : hipErrorInvalidValue;
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm(bool bf16, int epi, int mt, int nt, const GemmArgs& a, hipStream_t s) {
  if (nt != gemm_tiles(epi, mt, a.N) || a.wide_wgs != gemm_wide_wgs(epi, mt, a.N)) return hipErrorInvalidValue;
  if (a.ksplit != gemm_ksplit(epi, mt, a.N, a.nkc) || (a.ksplit > 1 && (!a.kpart || !a.kcount)))
    return hipErrorInvalidValue;
  if (bf16) {
    switch (mt) {
      case 1: return launch_rows<_Float16, 1>(epi, nt, a, s);
      case 2: return launch_rows<_Float16, 2>(epi, nt, a, s);
      case 3: return launch_rows<_Float16, 3>(epi, nt, a, s);
      case 4: return launch_rows<_Float16, 4>(epi, nt, a, s);
      case 5: return launch_rows<_Float16, 5>(epi, nt, a, s);
      case 6: return launch_rows<_Float16, 6>(epi, nt, a, s);
      case 7: return launch_rows<_Float16, 7>(epi, nt, a, s);
      case 8: return launch_rows<_Float16, 8>(epi, nt, a, s);
      default: return hipErrorInvalidValue;
    }
  }
  switch (mt) {
    case 1: return launch_rows<float, 1>(epi, nt, a, s);
    case 2: return launch_rows<float, 2>(epi, nt, a, s);
    case 3: return launch_rows<float, 3>(epi, nt, a, s);
    case 4: return launch_rows<float, 4>(epi, nt, a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tss
