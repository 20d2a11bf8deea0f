// Weight GEMMs of the decode loop: C[m][n] = sum_k X[m][k] * W[n][k].
//
// Weights are stored fragment-tiled (device_common.h): every wave load of a
// weight fragment is one contiguous 1 KB block, and the waves of a workgroup
// take interleaved k-fragments so that together they read one contiguous
// window.  Four matrix-core kernels share one set of fused epilogues:
//  * k_gemm_skinny (M <= 8 rows: decode, micro steps, LM head; up to 64 for
//    the embedder's output epilogues).  HBM-bound
//    weight streaming with non-temporal loads; four waves split the k-range of
//    a 16*TN-column tile, and loads of the next batch of fragments are issued
//    before the matrix instructions of the current one.  The k dimension may
//    also be split across workgroups: each split then writes fp32 partials
//    [split][M][N] and the consuming kernel sums them in split order (no
//    cross-workgroup synchronisation inside a kernel: on this GPU the L2 of one
//    XCD is not coherent with the others, and the write-back fences that a
//    handshake needs cost far more than a kernel boundary).
//  * k_gemm_staged (M <= 8): the skinny GEMM with eight waves whose X operand
//    is built in LDS by a prologue (an RMSNorm of the residual plus pending
//    partials, or the merge of the attention splits), so the kernel that
//    would produce X disappears from the launch sequence.
//  * k_gemm_wide (8 < M <= 256: batched decode, micro context rows): eight
//    waves own eight column tiles and share X chunks through LDS.
//  * k_gemm_big (larger M: prefill chunks): 128x128 LDS-staged tiles, double
//    buffered, 2x2 waves of 64x64.
// X rows are the A operand (padded to 16), weight rows the B operand, so the
// accumulator's columns are output features: lane l holds column l & 15 of a
// 16-column tile for rows 4*(l >> 4) + i.
#include <algorithm>
#include <type_traits>

#include "decide.h"
#include "device_common.h"
#include "ham_internal.h"

namespace ham {

// Epilogue of one accumulator element: row m, column nb + r16 of the tile at nb.
// Every lane must call it (the SwiGLU pairing exchanges values between lanes).
template <typename T, int EPI>
__device__ __forceinline__ void epi_tile(const GemmArgs& a, int m, bool ok, int nb, int r16, float v) {
  const int n = nb + r16;
  if constexpr (EPI == EPI_SWIGLU) {
    // a 16-row tile holds gate rows of 8 features then their up rows
    const float u = __shfl_xor(v, 8, WAVE);
    if (ok && r16 < 8) {
      const float sg = v / (1.0f + expf(-v));
      Act<T>::put(a.out, m, a.ldo, nb / 2 + r16, sg * u);
    }
  } else {
    if (!ok) return;
    if constexpr (EPI == EPI_F32) {
      ((float*)a.out)[(size_t)m * a.ldo + n] = v;
    } else if constexpr (EPI == EPI_OP) {
      Act<T>::put(a.out, m, a.ldo, n, v);
    } else if constexpr (EPI == EPI_RESID) {
      float* o = (float*)a.out + (size_t)m * a.ldo;
      o[n] += v;
    } else if constexpr (EPI == EPI_XMASK) {
      if (a.rowmask[m]) ((float*)a.out)[(size_t)m * a.ldo + n] = v;
    }
  }
}

__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

// ------------------------------------------------------------------------ skinny
template <typename T, int MT, int TN>
struct SkinnyBatch {
  static constexpr int U = 4;
  u4 w[U][TN];
  u4 xh[U][MT], xl[U][MT];
};

// fragment f of every operand: weight block (tile j, f) at wrow[j] + f*512 elements-of-16B
template <typename T, int MT, int TN>
__device__ __forceinline__ void skinny_load(SkinnyBatch<T, MT, TN>& b, const T* const* wrow, const T* const* xrow,
                                            const bool* xok, int lo_off, int f, int stride) {
  constexpr int KB = Frag<T>::KB, EPL = Frag<T>::EPL, U = SkinnyBatch<T, MT, TN>::U;
#pragma unroll
  for (int u = 0; u < U; ++u) {
#pragma unroll
    for (int j = 0; j < TN; ++j) b.w[u][j] = ld16_stream(wrow[j] + (size_t)(f + u * stride) * 64 * EPL);
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      // only lanes of live rows load (rows past M would fetch 1 KB per wave
      // instruction through the vector cache for nothing)
      b.xh[u][i] = zero16();
      b.xl[u][i] = zero16();
      if (xok[i]) {
        b.xh[u][i] = ld16(xrow[i] + (size_t)(f + u * stride) * KB);
        if constexpr (Act<T>::SPLIT) b.xl[u][i] = ld16(xrow[i] + lo_off + (size_t)(f + u * stride) * KB);
      }
    }
  }
}

template <typename T, int MT, int TN>
__device__ __forceinline__ void skinny_mma(f4 (*acc)[TN], const SkinnyBatch<T, MT, TN>& b) {
#pragma unroll
  for (int u = 0; u < SkinnyBatch<T, MT, TN>::U; ++u)
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) mma_act<T>(acc[i][j], b.xh[u][i], b.xl[u][i], b.w[u][j]);
}

template <typename T, int MT, int TN, int EPI, int NW>
__device__ __forceinline__ void skinny_finish(const GemmArgs& a, f4 (*acc)[TN], float* red, int ntile, int split,
                                              int nsplit, int n0);
template <typename T, int MT, int TN, int EPI>
__device__ __forceinline__ void skinny_epilogue(const GemmArgs& a, f4 (*acc)[TN], int ntile, int split, int nsplit,
                                                int n0);

// Reduction of the NW waves' k-slices of one workgroup into wave 0's
// accumulators (fixed order: wave 0, 1, ...; red holds [NW-1][NACC][64]
// floats).  Returns whether this wave holds the result (wave 0).
template <int MT, int TN, int NW>
__device__ __forceinline__ bool skinny_reduce(f4 (*acc)[TN], float* red) {
  constexpr int NACC = MT * TN * 4;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (w > 0) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[((w - 1) * NACC + (i * TN + j) * 4 + r) * 64 + lane] = acc[i][j][r];
  }
  __syncthreads();
  if (w != 0) return false;
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int q = (i * TN + j) * 4 + r;
        float v = acc[i][j][r];
#pragma unroll
        for (int p = 0; p < NW - 1; ++p) v += red[(p * NACC + q) * 64 + lane];
        acc[i][j][r] = v;
      }
  return true;
}

// Per-row sums over the n tiles of ss [n][M] (n <= NORM_OUT_MAX_TILES, rows
// m < M <= NORM_OUT_MAX_ROWS), wave-cooperative: lane l adds tiles l, l + 64,
// ... in order, then a butterfly over the wave (all loads are issued before
// the first is added).
struct TileSums {
  float p[NORM_OUT_MAX_ROWS];
};
__device__ __forceinline__ void tile_sums_load(TileSums& t, const float* ss, int n, int M) {
  const int lane = threadIdx.x & 63;
  constexpr int Q = NORM_OUT_MAX_TILES / 64;
  float v[Q][NORM_OUT_MAX_ROWS];
#pragma unroll
  for (int q = 0; q < Q; ++q)
#pragma unroll
    for (int m = 0; m < NORM_OUT_MAX_ROWS; ++m) {
      const int tt = lane + 64 * q;
      v[q][m] = (tt < n && m < M) ? ss[(size_t)tt * M + m] : 0.f;
    }
#pragma unroll
  for (int m = 0; m < NORM_OUT_MAX_ROWS; ++m) {
    float acc = 0.f;
#pragma unroll
    for (int q = 0; q < Q; ++q) acc += v[q][m];
    t.p[m] = acc;
  }
}

// Row scale 1/rms of this lane's rows 4g + r (MT = 1: rows below 16; rows past
// NORM_OUT_MAX_ROWS keep 1, they are never stored)
__device__ __forceinline__ void tile_sums_rinv(const TileSums& t, const RowScale& rs, float (&sc)[4]) {
  const int g = (threadIdx.x & 63) >> 4;
  float rin[NORM_OUT_MAX_ROWS];
#pragma unroll
  for (int m = 0; m < NORM_OUT_MAX_ROWS; ++m) rin[m] = 1.0f / sqrtf(wave_sum(t.p[m]) / (float)rs.d + rs.eps);
  static_assert(NORM_OUT_MAX_ROWS == 8, "rows of lane groups 0 and 1");
#pragma unroll
  for (int r = 0; r < 4; ++r) sc[r] = g == 0 ? rin[r] : (g == 1 ? rin[4 + r] : 1.f);
}

// The NormOut epilogue of wave 0 (rows 4g + r, columns n0 + 16j + r16; MT = 1):
// x += product, optional copy to ctx, g * x as the next operand, and per row
// the sum of squares of this tile's columns.  xv holds x and gv the gain,
// loaded at the start of the kernel.
template <typename T, int TN>
__device__ __forceinline__ void norm_out_epilogue(const GemmArgs& a, f4 (*acc)[TN], const float (*xv)[4],
                                                  const float* gv, int ntile, int n0) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, g = lane >> 4;
  float sq[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = 4 * g + r, n = n0 + 16 * j + r16;
      if (m < a.M) {
        const float x = xv[j][r] + acc[0][j][r];
        ((float*)a.out)[(size_t)m * a.ldo + n] = x;
        if (a.ctx) a.ctx[(size_t)m * a.ldctx + n] = x;
        if (a.no.g) Act<T>::put(a.no.act, m, a.no.lda, n, gv[j] * x);
        sq[r] += x * x;
      }
    }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float v = sq[r];
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1) v += __shfl_xor(v, o, WAVE);  // the 16 columns of lane group g
    const int m = 4 * g + r;
    if (r16 == 0 && m < a.M) a.no.ss[(size_t)ntile * a.M + m] = v;
  }
}

// TAG only separates the names of base-layer launches (always active) from the
// others in profiler output; the code is the same.  NW waves split the k-range
// of the tile (4, or 16 for the unsplit NormOut launch: one workgroup per tile).
template <typename T, int MT, int TN, int EPI, int TAG, int NW = 4>
__global__ __launch_bounds__(64 * NW) void k_gemm_skinny(GemmArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  constexpr int EPL = Frag<T>::EPL, KB = Frag<T>::KB;
  constexpr int NACC = MT * TN * 4;
  constexpr int U = SkinnyBatch<T, MT, TN>::U;
  __shared__ float red[NW - 1][NACC][64];  // k-slices of waves 1..NW-1
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int ntile = blockIdx.x, split = blockIdx.y, nsplit = gridDim.y;
  const int n0 = ntile * 16 * TN;
  const int nfr = a.K / KB;
  const int c0 = (int)((long)split * nfr / nsplit), c1 = (int)((long)(split + 1) * nfr / nsplit);
  // wave w takes fragments c0 + w + NW i of the k-range: at any moment the
  // waves read neighbouring 1 KB blocks of a tile (one contiguous window)
  const int nk = c1 - c0, cnt = nk > w ? (nk - w + NW - 1) / NW : 0;
  const T* W = (const T*)a.W;
  const T* X = (const T*)a.X;

  f4 acc[MT][TN];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  // NormOut launch: wave 0 loads the residual values and gains its epilogue
  // needs before any weight load (used only at the end, they wait for nothing)
  constexpr bool NORM_OUT = NW == 16;
  static_assert(!NORM_OUT || (EPI == EPI_RESID && MT == 1), "NormOut: RESID, rows below 16");
  float xv[TN][4], gv[TN];
  if constexpr (NORM_OUT) {
    if (w == 0) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int n = n0 + 16 * j + r16;
        gv[j] = a.no.g ? a.no.g[n] : 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = 4 * g + r;
          xv[j][r] = m < a.M ? ((const float*)a.out)[(size_t)m * a.ldo + n] : 0.f;
        }
      }
    }
  }

  const T* wrow[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) wrow[j] = W + (size_t)(n0 / 16 + j) * nfr * 64 * EPL + (size_t)lane * EPL;
  constexpr int PL = Act<T>::PL;
  const int lo_off = Act<T>::SPLIT ? a.ldx : 0;  // offset of the lo plane within a row
  const T* xrow[MT];
  bool xok[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int m = 16 * i + r16;
    xok[i] = m < a.M;
    xrow[i] = X + (size_t)(xok[i] ? m : 0) * a.ldx * PL + g * EPL;
  }

  // software pipeline over batches of U fragments: the loads of batch i+1 are
  // in flight while batch i feeds the matrix cores
  const int nb = cnt / U;
  SkinnyBatch<T, MT, TN> cur, nxt;
  if (nb > 0) skinny_load<T, MT, TN>(cur, wrow, xrow, xok, lo_off, c0 + w, NW);
  for (int it = 0; it < nb; ++it) {
    const bool more = it + 1 < nb;
    if (more) skinny_load<T, MT, TN>(nxt, wrow, xrow, xok, lo_off, c0 + w + NW * (it + 1) * U, NW);
    skinny_mma<T, MT, TN>(acc, cur);
    if (more) cur = nxt;
  }
  for (int i = nb * U; i < cnt; ++i) {
    const int f = c0 + w + NW * i;
    u4 bw[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) bw[j] = ld16_stream(wrow[j] + (size_t)f * 64 * EPL);
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      u4 h = zero16(), l = zero16();
      if (xok[i]) {
        h = ld16(xrow[i] + (size_t)f * KB);
        if constexpr (Act<T>::SPLIT) l = ld16(xrow[i] + lo_off + (size_t)f * KB);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) mma_act<T>(acc[i][j], h, l, bw[j]);
    }
  }

  if constexpr (NORM_OUT) {
    if (skinny_reduce<MT, TN, NW>(acc, &red[0][0][0])) norm_out_epilogue<T, TN>(a, acc, xv, gv, ntile, n0);
  } else if constexpr (EPI == EPI_SWIGLU && MT == 1) {
    // rows scaled by 1/rms before the activation: wave 0 issues the loads of
    // the tile sums before the cross-wave reduction waits on the other waves
    // (issued with the first weights instead, the compiler's waits for them
    // held back the weight stream: measured no faster)
    TileSums ts;
    if (a.rs.ss && w == 0) tile_sums_load(ts, a.rs.ss, a.rs.n, a.M);
    if (skinny_reduce<MT, TN, NW>(acc, &red[0][0][0])) {
      if (a.rs.ss) {
        float sc[4];
        tile_sums_rinv(ts, a.rs, sc);
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[0][j][r] *= sc[r];
      }
      skinny_epilogue<T, MT, TN, EPI>(a, acc, ntile, split, nsplit, n0);
    }
  } else {
    skinny_finish<T, MT, TN, EPI, NW>(a, acc, &red[0][0][0], ntile, split, nsplit, n0);
  }
}

// Reduction of the NW waves' k-slices and the epilogue: split partials, the
// LM head's per-tile argmax, or the fused epilogue.
template <typename T, int MT, int TN, int EPI, int NW>
__device__ __forceinline__ void skinny_finish(const GemmArgs& a, f4 (*acc)[TN], float* red, int ntile, int split,
                                              int nsplit, int n0) {
  if (skinny_reduce<MT, TN, NW>(acc, red)) skinny_epilogue<T, MT, TN, EPI>(a, acc, ntile, split, nsplit, n0);
}

// Epilogue of one wave's finished accumulators (rows 16i + 4g + r, columns
// n0 + 16j + r16): split partials, the LM head's per-tile argmax, or the fused epilogue.
template <typename T, int MT, int TN, int EPI>
__device__ __forceinline__ void skinny_epilogue(const GemmArgs& a, f4 (*acc)[TN], int ntile, int split, int nsplit,
                                                int n0) {
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, g = lane >> 4;
  if (nsplit > 1) {  // partial of this k-chunk; the consumer sums the chunks in order
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = 16 * i + 4 * g + r;
          if (m < a.M) a.part[((size_t)split * a.M + m) * a.N + n0 + 16 * j + r16] = acc[i][j][r];
        }
    return;
  }

  if constexpr (EPI == EPI_ARGMAX) {
    // per-row best (value, lowest index) of this column tile; the stop-head row V
    // is kept aside; k_decide finishes the argmax over all tiles
    const DecideArgs& d = a.dec;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = 16 * i + 4 * g + r;
        float bv = -INFINITY;
        int bi = 0x7fffffff;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int n = n0 + 16 * j + r16;
          const float v = acc[i][j][r];
          if (m < a.M) {
            if (n < d.V) {
              if (better(v, n, bv, bi)) { bv = v; bi = n; }
              if (d.dbg_logits) d.dbg_logits[(size_t)m * d.V + n] = v;
            } else if (n == d.V) {
              d.stop_buf[m] = v;
            }
          }
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          const float ov = __shfl_xor(bv, o, WAVE);
          const int oi = __shfl_xor(bi, o, WAVE);
          if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
        }
        if (r16 == 0 && m < a.M) {
          d.best_val[(size_t)m * d.ntiles + ntile] = bv;
          d.best_idx[(size_t)m * d.ntiles + ntile] = bi;
        }
      }
  } else {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = 16 * i + 4 * g + r;
          epi_tile<T, EPI>(a, m, m < a.M, n0 + 16 * j, r16, acc[i][j][r]);
        }
  }
}


// ------------------------------------------------------------------------ staged
// Skinny GEMM whose X operand is built in LDS by a prologue (XStage): eight
// waves split the k-range of a 16*TN-column tile; the first batch of weight
// loads is issued before the prologue so both are in flight together.
// Rows M <= 8 and M * (k-range) <= STG_VALS values.
constexpr int STG_NW = 8;
constexpr int STG_THREADS = 64 * STG_NW;
constexpr int STG_CH = 2;                         // 4-value chunks of X per thread
constexpr int STG_VALS = STG_CH * STG_THREADS * 4;  // X values one workgroup stages
constexpr int STG_SMAX = 8;                       // pending partials summed by the NORM prologue
constexpr int STG_AMAX = 8;                       // attention splits one thread combines
constexpr int STG_MMAX = 8;

// 4 consecutive values of X row m at local column kl -> the LDS operand layout
// (bf16: hi plane then lo plane per row, 4 bytes per value in total; fp32: as is)
template <typename T>
__device__ __forceinline__ void stage_put4(char* stg, int Kr, int m, int kl, f4 v);
template <>
__device__ __forceinline__ void stage_put4<bf16>(char* stg, int Kr, int m, int kl, f4 v) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bf16 hb = f2bf(v[e]);
    h[e] = hb;
    l[e] = f2bf(v[e] - bf2f(hb));
  }
  char* row = stg + (size_t)m * 4 * Kr;
  *reinterpret_cast<uint2*>(row + (size_t)kl * 2) = uint2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
  *reinterpret_cast<uint2*>(row + (size_t)2 * Kr + (size_t)kl * 2) = uint2{l[0] | (l[1] << 16), l[2] | (l[3] << 16)};
}
template <>
__device__ __forceinline__ void stage_put4<float>(char* stg, int Kr, int m, int kl, f4 v) {
  *reinterpret_cast<f4*>(stg + (size_t)m * 4 * Kr + (size_t)kl * 4) = v;
}

// XS_NORM prologue.  Chunk i (of M * Kr/4) is row i / (Kr/4), columns k0 + 4*(i % (Kr/4)).
// aux: [nch] chunk sums of squares, then [M] row sums.
// The prologue's global loads come first in the kernel, ahead of the first
// weight blocks: loads of one wave return in issue order, so prologue data
// issued after the weights would wait for them.
struct NormLoads {
  f4 v[STG_CH], gv[STG_CH];
  f4 pv[STG_CH][STG_SMAX];
};
__device__ __forceinline__ void stage_norm_load(const GemmArgs& a, NormLoads& L, int k0, int Kr) {
  const XStage& s = a.xs;
  const int tid = threadIdx.x;
  const int M = a.M, cpr = Kr / 4, nch = M * cpr;
  const int ns = s.part ? s.nsplit : 0;
  // only the needed loads issue (every vector memory instruction costs address
  // cycles for its active lanes, whether or not it fetches anything)
#pragma unroll
  for (int j = 0; j < STG_CH; ++j) {
    const int i = tid + j * STG_THREADS;
    if (i < nch) {
      const int m = i / cpr, k = k0 + (i % cpr) * 4;
      L.v[j] = *reinterpret_cast<const f4*>(s.x + (size_t)m * s.ldx + k);
      L.gv[j] = *reinterpret_cast<const f4*>(s.g + k);
#pragma unroll
      for (int q = 0; q < STG_SMAX; ++q)
        if (q < ns) L.pv[j][q] = *reinterpret_cast<const f4*>(s.part + ((size_t)q * s.pM + m) * s.ldx + k);
    }
  }
}

// The summed residual (and the context copy, and the k-range's sums of squares
// when the k-range is split) leave the workgroup later, in stage_norm_publish:
// a global store in flight makes every later wait for a load a wait for all of
// them (stores and loads share one counter here), prefetched weights included.
template <typename T>
__device__ __forceinline__ void stage_norm(const GemmArgs& a, NormLoads& L, char* stg, float* aux, int k0, int Kr) {
  const XStage& s = a.xs;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int M = a.M, cpr = Kr / 4, nch = M * cpr;
  const int ns = s.part ? s.nsplit : 0;
  const bool whole = gridDim.y == 1;  // the workgroup sees whole rows: apply rinv here
  f4* v = L.v;
  f4* gv = L.gv;
  f4 (*pv)[STG_SMAX] = L.pv;
  float* sq = aux;
  float* ssr = aux + nch;
#pragma unroll
  for (int j = 0; j < STG_CH; ++j) {
    const int i = tid + j * STG_THREADS;
    if (i < nch) {
#pragma unroll
      for (int q = 0; q < STG_SMAX; ++q)
        if (q < ns) v[j] += pv[j][q];
      const f4 x = v[j];
      sq[i] = (x[0] * x[0] + x[1] * x[1]) + (x[2] * x[2] + x[3] * x[3]);
    }
  }
  lds_barrier();
  if (w < M) {  // wave m: the sum of squares of row m over this k-range, fixed order
    float t = 0.f;
    for (int c = lane; c < cpr; c += 64) t += sq[w * cpr + c];
    t = wave_sum(t);
    if (lane == 0) ssr[w] = t;
  }
  lds_barrier();
#pragma unroll
  for (int j = 0; j < STG_CH; ++j) {
    const int i = tid + j * STG_THREADS;
    if (i < nch) {
      const int m = i / cpr, kl = (i % cpr) * 4;
      const float sc = whole ? 1.0f / sqrtf(ssr[m] / (float)a.K + s.eps) : 1.0f;
      stage_put4<T>(stg, Kr, m, kl, v[j] * sc * gv[j]);
    }
  }
}

// Column tile 0's workgroup of each k-range writes the summed residual rows (and
// the context copy) and, when the k-range is split, the range's sums of squares.
__device__ __forceinline__ void stage_norm_publish(const GemmArgs& a, const NormLoads& L, const float* aux, int k0,
                                                   int Kr, int split) {
  const XStage& s = a.xs;
  const int tid = threadIdx.x;
  const int M = a.M, cpr = Kr / 4, nch = M * cpr;
#pragma unroll
  for (int j = 0; j < STG_CH; ++j) {
    const int i = tid + j * STG_THREADS;
    if (i < nch) {
      const int m = i / cpr, k = k0 + (i % cpr) * 4;
      *reinterpret_cast<f4*>(s.x_out + (size_t)m * s.ldx + k) = L.v[j];
      if (s.ctx) *reinterpret_cast<f4*>(s.ctx + (size_t)m * s.ldctx + k) = L.v[j];
    }
  }
  if (gridDim.y > 1 && tid < M) s.ss_out[(size_t)split * M + tid] = aux[nch + tid];
}

// XS_ATTN prologue.  Heads h0.. of the k-range; one wave per (row, head)
// forms the softmax weights exp(m_s - M) / L of the splits (lane s holds split
// s), then thread (chunk c, group sg) sums the weighted outputs of splits sg,
// sg + SG, ... and the groups are added in order.  aux: [M][nh][ans] weights,
// then [SG][nch] 4-value partial sums.
struct AttnLoads {
  f4 o[STG_AMAX];   // the split outputs this thread combines
  float ms0, ls0;   // (max, sum) of split `lane` for this wave's first (row, head)
};
__device__ __forceinline__ void stage_attn_load(const GemmArgs& a, AttnLoads& L, int k0, int Kr) {
  const XStage& s = a.xs;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int M = a.M, hd = s.hd, ans = s.ans, grp = s.grp, Hkv = s.Hkv;
  const int h0 = k0 / hd, nh = (k0 + Kr - 1) / hd + 1 - h0;
  const int cpr = Kr / 4, nch = M * cpr;
  const int SG = max(1, min(STG_THREADS / nch, ans));
  const int c = tid % nch, sg = tid / nch;
  const bool act = tid < nch * SG;
  const int m = c / cpr, k = k0 + (c % cpr) * 4, h = k / hd, d = k % hd;
  if (act) {
    const float* ob = s.rec_o + ((((size_t)m * Hkv + h / grp) * ans) * grp + h % grp) * hd + d;
#pragma unroll
    for (int q = 0; q < STG_AMAX; ++q) {
      const int sp = sg + q * SG;
      if (sp < ans) L.o[q] = *reinterpret_cast<const f4*>(ob + (size_t)sp * grp * hd);
    }
  }
  L.ms0 = -INFINITY;
  L.ls0 = 0.f;
  if (w < M * nh && lane < ans) {
    const int gm = w / nh, gh = h0 + w % nh;
    const size_t q = (((size_t)gm * Hkv + gh / grp) * ans + lane) * grp + gh % grp;
    L.ms0 = s.rec_ml[2 * q];
    L.ls0 = s.rec_ml[2 * q + 1];
  }
}

template <typename T>
__device__ __forceinline__ void stage_attn(const GemmArgs& a, AttnLoads& L, char* stg, float* aux, int k0, int Kr) {
  const XStage& s = a.xs;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int M = a.M, hd = s.hd, ans = s.ans, grp = s.grp, Hkv = s.Hkv;
  const int h0 = k0 / hd, nh = (k0 + Kr - 1) / hd + 1 - h0;
  const int cpr = Kr / 4, nch = M * cpr;
  const int SG = max(1, min(STG_THREADS / nch, ans));
  float* wts = aux;
  f4* ps = reinterpret_cast<f4*>(aux + ((M * nh * ans + 3) & ~3));
  const int c = tid % nch, sg = tid / nch;
  const bool act = tid < nch * SG;
  const int m = c / cpr, k = k0 + (c % cpr) * 4, h = k / hd, d = k % hd;
  f4* o = L.o;
  for (int gi = w; gi < M * nh; gi += STG_NW) {
    const int gm = gi / nh, gh = h0 + gi % nh;
    float ms = -INFINITY, ls = 0.f;
    if (gi == w) {
      if (lane < ans) {
        ms = L.ms0;
        ls = L.ls0;
      }
    } else if (lane < ans) {
      const size_t q = (((size_t)gm * Hkv + gh / grp) * ans + lane) * grp + gh % grp;
      ms = s.rec_ml[2 * q];
      ls = s.rec_ml[2 * q + 1];
    }
    const float Mx = wave_max(ms);
    const float e = (ms == -INFINITY) ? 0.f : __expf(ms - Mx);
    const float L = wave_sum(e * ls);
    if (lane < ans) wts[gi * ans + lane] = L > 0.f ? e / L : 0.f;
  }
  lds_barrier();
  if (act) {
    const float* wt = wts + (m * nh + (h - h0)) * ans;
    f4 acc = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < STG_AMAX; ++q) {
      const int sp = sg + q * SG;
      if (sp < ans) acc += wt[sp] * o[q];
    }
    ps[tid] = acc;
  }
  lds_barrier();
  for (int i = tid; i < nch; i += STG_THREADS) {
    f4 x = ps[i];
    for (int q = 1; q < SG; ++q) x += ps[q * nch + i];
    stage_put4<T>(stg, Kr, i / cpr, (i % cpr) * 4, x);
  }
}

// LDS bytes of a staged launch: wave reduction, X rows, prologue scratch
__host__ __device__ inline size_t stage_lds_bytes(int tn, int M, int Kr, int xsrc, int ans, int hd) {
  const size_t red = (size_t)(STG_NW - 1) * tn * 4 * 64 * 4;
  const size_t stg = (size_t)M * Kr * 4;
  const int nch = M * Kr / 4;
  size_t aux;
  if (xsrc == XS_NORM) {
    aux = (size_t)(nch + STG_MMAX) * 4;
  } else {
    const int nh = Kr / hd + 2, nml = M * nh * ans;
    aux = (size_t)((nml + 3) & ~3) * 4 + (size_t)STG_THREADS * 16;
  }
  return red + stg + aux;
}

template <typename T, int TN, int EPI, int TAG, int XS>
__global__ __launch_bounds__(STG_THREADS) void k_gemm_staged(GemmArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  constexpr int EPL = Frag<T>::EPL, KB = Frag<T>::KB, U = 4;
  extern __shared__ float dsm[];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int ntile = blockIdx.x, split = blockIdx.y, nsplit = gridDim.y;
  const int n0 = ntile * 16 * TN;
  const int nfr = a.K / KB;
  const int c0 = (int)((long)split * nfr / nsplit), c1 = (int)((long)(split + 1) * nfr / nsplit);
  const int Kr = (c1 - c0) * KB;
  // wave w takes fragments c0 + w + STG_NW*i of the k-range: at any moment the
  // waves of a workgroup read neighbouring 1 KB blocks of a tile
  const int nk = c1 - c0, cnt = nk > w ? (nk - w + STG_NW - 1) / STG_NW : 0;
  const auto FR = [&](int i) { return c0 + w + STG_NW * i; };
  float* red = dsm;
  char* stg = reinterpret_cast<char*>(dsm + (STG_NW - 1) * TN * 4 * 64);
  float* aux = reinterpret_cast<float*>(stg + (size_t)a.M * 4 * Kr);
  const T* W = (const T*)a.W;
  const T* wrow[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) wrow[j] = W + (size_t)(n0 / 16 + j) * nfr * 64 * EPL + (size_t)lane * EPL;
  // the prologue's loads, then the wave's first PF weight fragments, are in
  // flight before the prologue computes (8 weight blocks in all: more would
  // cost the occupancy of two workgroups per CU)
  typename std::conditional<XS == XS_NORM, NormLoads, AttnLoads>::type pl;
  if constexpr (XS == XS_NORM) stage_norm_load(a, pl, c0 * KB, Kr);
  else stage_attn_load(a, pl, c0 * KB, Kr);
  __builtin_amdgcn_sched_barrier(0);
  constexpr int PF = 8 / TN;
  const int npf = min(PF, cnt);
  u4 wp[PF][TN];
  {  // range-checked: blocks past this wave's k-range read zeros, fetch nothing
    const BufRsrc rw = buf_rsrc(W, (uint32_t)((size_t)a.N * a.K * sizeof(T)));
#pragma unroll
    for (int u = 0; u < PF; ++u)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        wp[u][j] = buf_u4_stream(rw, u < npf ? (uint32_t)(((size_t)(n0 / 16 + j) * nfr + FR(u)) * 64 * EPL +
                                                          (size_t)lane * EPL) * (uint32_t)sizeof(T)
                                             : BUF_OOB);
  }
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (XS == XS_NORM) stage_norm<T>(a, pl, stg, aux, c0 * KB, Kr);
  else stage_attn<T>(a, pl, stg, aux, c0 * KB, Kr);
  lds_barrier();
  const int i0 = npf;
  const int nb = (cnt - i0) / U;
  u4 wc[U][TN], wn[U][TN];
  auto wload = [&](u4 (*dst)[TN], int i) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < TN; ++j) dst[u][j] = ld16_stream(wrow[j] + (size_t)FR(i + u) * 64 * EPL);
  };
  const bool xrow = r16 < a.M;
  const char* xb = stg + (size_t)(xrow ? r16 : 0) * 4 * Kr + (size_t)g * EPL * sizeof(T);
  auto xfrag = [&](int f, u4& h, u4& l) {
    const char* p = xb + (size_t)(f - c0) * KB * sizeof(T);
    h = xrow ? *reinterpret_cast<const u4*>(p) : zero16();
    l = (Act<T>::SPLIT && xrow) ? *reinterpret_cast<const u4*>(p + 2 * Kr) : zero16();
  };
  f4 acc[1][TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) acc[0][j] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < PF; ++u)
    if (u < npf) {
      u4 h, l;
      xfrag(FR(u), h, l);
#pragma unroll
      for (int j = 0; j < TN; ++j) mma_act<T>(acc[0][j], h, l, wp[u][j]);
    }
  // the rest in batches of U; issuing the first batch only once the prefetched
  // blocks have arrived measured faster than issuing it right after the prologue
  if (nb > 0) wload(wc, i0);
  for (int it = 0; it < nb; ++it) {
    const bool more = it + 1 < nb;
    if (more) wload(wn, i0 + (it + 1) * U);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      u4 h, l;
      xfrag(FR(i0 + it * U + u), h, l);
#pragma unroll
      for (int j = 0; j < TN; ++j) mma_act<T>(acc[0][j], h, l, wc[u][j]);
    }
    if (more) {
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < TN; ++j) wc[u][j] = wn[u][j];
    }
  }
  for (int i = i0 + nb * U; i < cnt; ++i) {
    const int f = FR(i);
    u4 bw[TN], h, l;
#pragma unroll
    for (int j = 0; j < TN; ++j) bw[j] = ld16_stream(wrow[j] + (size_t)f * 64 * EPL);
    xfrag(f, h, l);
#pragma unroll
    for (int j = 0; j < TN; ++j) mma_act<T>(acc[0][j], h, l, bw[j]);
  }
  if constexpr (XS == XS_NORM)
    if (ntile == 0) stage_norm_publish(a, pl, aux, c0 * KB, Kr, split);
  skinny_finish<T, 1, TN, EPI, STG_NW>(a, acc, red, ntile, split, nsplit, n0);
}

// ------------------------------------------------------------------------ wide
// Batched skinny GEMM (8 < M <= 256 rows): a workgroup of eight waves owns eight
// column tiles of 16*TN columns (one per wave) and one k-range.  The X rows of
// the k-range pass through LDS in chunks of WIDE_KC columns shared by the eight
// waves, so a workgroup reads X once for eight tiles instead of once per tile;
// each wave streams its own weight blocks with the next chunk in flight.  Waves
// own disjoint columns, so there is no cross-wave reduction.
constexpr int WIDE_NW = 8;
constexpr int WIDE_KC = 128;
constexpr int MAX_WIDE_SWIGLU_SPLIT = 4;

// NX: X is the RMSNorm of fp32 rows whose sums of squares the norm's first
// phase left in 256-column chunks (XS_NORMW): each staged chunk is scaled by
// the row's 1/rms and the gain and split into the operand planes here, in the
// order and precision the norm's second phase would use.
template <typename T, int MT, int TN, int EPI, int TAG, bool NX = false>
__global__ __launch_bounds__(64 * WIDE_NW) void k_gemm_wide(GemmArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  constexpr int KC = MT <= 4 ? WIDE_KC : WIDE_KC / 2;  // k per chunk: LDS holds two chunks of all rows
  constexpr int EPL = Frag<T>::EPL, KB = Frag<T>::KB, FPC = KC / KB;
  constexpr int PL = Act<T>::PL;
  constexpr int ROWB = KC * (int)sizeof(T) + 16;  // one row-plane of a chunk, padded against bank conflicts
  constexpr int RT = MT * 16;
  constexpr int PIECES = KC * (int)sizeof(T) / 16;
  constexpr int ITEMS = RT * PL * PIECES;
  constexpr int IPT = (ITEMS + 64 * WIDE_NW - 1) / (64 * WIDE_NW);
  __shared__ __align__(16) char xs[2][RT][PL][ROWB];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int ntiles = a.N / (16 * TN);
  const int ntile = blockIdx.x * WIDE_NW + w;
  const bool tile_ok = ntile < ntiles;
  const int n0 = ntile * 16 * TN;
  const int split = blockIdx.y, nsplit = gridDim.y;
  const int nfr = a.K / KB, nch = a.K / KC;
  const int ch0 = (int)((long)split * nch / nsplit), ch1 = (int)((long)(split + 1) * nch / nsplit);
  const T* W = (const T*)a.W;
  const T* X = (const T*)a.X;
  const T* wrow[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j)  // a wave past the last tile streams the last tile's blocks (never used)
    wrow[j] = W + (size_t)((tile_ok ? ntile : ntiles - 1) * TN + j) * nfr * 64 * EPL + (size_t)lane * EPL;

  constexpr int Q4 = KC / 4;                                   // NX: 4-value pieces per row of a chunk
  constexpr int IPTN = NX ? (RT * Q4 + 64 * WIDE_NW - 1) / (64 * WIDE_NW) : 1;
  __shared__ float rinv_s[NX ? RT : 1];
  u4 xr[NX ? 1 : IPT];
  f4 xv[IPTN], xg[IPTN];
  auto xload = [&](int c) {
    if constexpr (NX) {
#pragma unroll
      for (int q = 0; q < IPTN; ++q) {
        const int i = tid + q * 64 * WIDE_NW;
        xv[q] = f4{0.f, 0.f, 0.f, 0.f};
        xg[q] = f4{0.f, 0.f, 0.f, 0.f};
        if (i < RT * Q4) {
          const int m = i / Q4, col = c * KC + (i % Q4) * 4;
          xg[q] = *reinterpret_cast<const f4*>(a.xs.g + col);
          if (m < a.M) xv[q] = *reinterpret_cast<const f4*>(a.xs.x + (size_t)m * a.xs.ldx + col);
        }
      }
    } else {
#pragma unroll
      for (int q = 0; q < IPT; ++q) {
        const int i = tid + q * 64 * WIDE_NW;
        xr[q] = zero16();
        if (i < ITEMS) {
          const int m = i / (PL * PIECES), p = (i / PIECES) % PL, pc = i % PIECES;
          if (m < a.M) xr[q] = ld16(X + ((size_t)m * PL + p) * a.ldx + (size_t)c * KC + pc * (16 / (int)sizeof(T)));
        }
      }
    }
  };
  auto xstore = [&](int buf) {
    if constexpr (NX) {
#pragma unroll
      for (int q = 0; q < IPTN; ++q) {
        const int i = tid + q * 64 * WIDE_NW;
        if (i < RT * Q4) {
          const int m = i / Q4, k4 = (i % Q4) * 4;
          const float inv = rinv_s[m];
          f4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = xv[q][e] * inv * xg[q][e];
          if constexpr (Act<T>::SPLIT) {
            uint32_t h[4], l[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const bf16 hb = f2bf(v[e]);
              h[e] = hb;
              l[e] = f2bf(v[e] - bf2f(hb));
            }
            *reinterpret_cast<uint2*>(&xs[buf][m][0][k4 * 2]) = uint2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
            *reinterpret_cast<uint2*>(&xs[buf][m][PL - 1][k4 * 2]) = uint2{l[0] | (l[1] << 16), l[2] | (l[3] << 16)};
          } else {
            *reinterpret_cast<f4*>(&xs[buf][m][0][k4 * 4]) = v;
          }
        }
      }
    } else {
#pragma unroll
      for (int q = 0; q < IPT; ++q) {
        const int i = tid + q * 64 * WIDE_NW;
        if (i < ITEMS) {
          const int m = i / (PL * PIECES), p = (i / PIECES) % PL, pc = i % PIECES;
          *reinterpret_cast<u4*>(&xs[buf][m][p][pc * 16]) = xr[q];
        }
      }
    }
  };
  if constexpr (NX) {  // each row's 1/rms from the chunk sums, summed in chunk order
    for (int m = tid; m < RT; m += 64 * WIDE_NW) {
      float t = 0.f;
      if (m < a.M)
        for (int c = 0; c < a.xs.nchw; ++c) t += a.xs.ssw[(size_t)m * a.xs.nchw + c];
      rinv_s[m] = m < a.M ? 1.0f / sqrtf(t / (float)a.K + a.xs.eps) : 0.f;
    }
    __syncthreads();
  }
  u4 wa[FPC][TN], wb[FPC][TN];
  auto wload = [&](u4 (*dst)[TN], int c) {
#pragma unroll
    for (int f = 0; f < FPC; ++f)
#pragma unroll
      for (int j = 0; j < TN; ++j) dst[f][j] = ld16_stream(wrow[j] + (size_t)(c * FPC + f) * 64 * EPL);
  };
  f4 acc[MT][TN];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  if (ch0 < ch1) {
    xload(ch0);
    wload(wa, ch0);
    xstore(0);
  }
  __syncthreads();
  for (int c = ch0; c < ch1; ++c) {
    const int buf = (c - ch0) & 1;
    const bool more = c + 1 < ch1;
    if (more) {
      xload(c + 1);
      wload(wb, c + 1);
    }
#pragma unroll
    for (int f = 0; f < FPC; ++f) {
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const char* xp = &xs[buf][i * 16 + r16][0][(f * KB + g * EPL) * (int)sizeof(T)];
        const u4 h = *reinterpret_cast<const u4*>(xp);
        const u4 l = Act<T>::SPLIT ? *reinterpret_cast<const u4*>(xp + ROWB) : zero16();
#pragma unroll
        for (int j = 0; j < TN; ++j) mma_act<T>(acc[i][j], h, l, wa[f][j]);
      }
    }
    if (more) {
      xstore(buf ^ 1);
#pragma unroll
      for (int f = 0; f < FPC; ++f)
#pragma unroll
        for (int j = 0; j < TN; ++j) wa[f][j] = wb[f][j];
    }
    __syncthreads();
  }
  if (tile_ok) skinny_epilogue<T, MT, TN, EPI>(a, acc, ntile, split, nsplit, n0);
}

// Final argmax of one row over all column tiles (fixed total order: larger value,
// then lower index), then the decision and stop test of that sequence, then
// (a sequence still running) the input rows of the next micro step, so no
// separate launch prepares them.  Each thread issues all of its tile loads
// before comparing any of them.
constexpr int DECIDE_THREADS = 1024;
constexpr int DECIDE_PER = 8;  // tiles per thread: ntiles <= 8192

template <typename T>
__global__ __launch_bounds__(DECIDE_THREADS) void k_decide(DecideArgs d, int ntiles) {
  if (!any_flag(d.st.active, d.B)) return;
  __shared__ float sv[DECIDE_THREADS / 64];
  __shared__ int si[DECIDE_THREADS / 64];
  __shared__ int s_run, s_tok;
  const int m = blockIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  float v[DECIDE_PER];
  int ix[DECIDE_PER];
#pragma unroll
  for (int q = 0; q < DECIDE_PER; ++q) {
    const int t = threadIdx.x + q * DECIDE_THREADS;
    v[q] = -INFINITY;
    ix[q] = 0x7fffffff;
    if (t < ntiles) {
      v[q] = d.best_val[(size_t)m * ntiles + t];
      ix[q] = d.best_idx[(size_t)m * ntiles + t];
    }
  }
  float bv = -INFINITY;
  int bi = 0x7fffffff;
#pragma unroll
  for (int q = 0; q < DECIDE_PER; ++q)
    if (better(v[q], ix[q], bv, bi)) { bv = v[q]; bi = ix[q]; }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const float ov = __shfl_xor(bv, o, WAVE);
    const int oi = __shfl_xor(bi, o, WAVE);
    if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
  }
  if (lane == 0) {
    sv[w] = bv;
    si[w] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int q = 1; q < DECIDE_THREADS / 64; ++q)
      if (better(sv[q], si[q], bv, bi)) { bv = sv[q]; bi = si[q]; }
    decide_one(d, m, bi, d.stop_buf[m]);
    s_run = d.st.active[m];                    // this thread's own writes
    s_tok = s_run ? d.st.grp_tok[m * 4 + d.prep_k - 1] : 0;
  }
  __syncthreads();
  if (d.prep_k == 0 || !s_run) return;
  // rows [ctx_1..ctx_C, E[t]] (step 1) or [E[t]]: 4-value chunks, every load of
  // a batch in flight before its stores
  const T* E = (const T*)d.E + (size_t)s_tok * d.d;
  const int nc = d.prep_k == 1 ? d.C : 0;
  const float* ctx = d.ctx + (size_t)m * d.C * d.d;
  float* x = d.x + (size_t)m * (nc + 1) * d.d;
  const int cpr = d.d / 4, total = (nc + 1) * cpr;
  constexpr int PB = 4;
  for (int i0 = threadIdx.x; i0 < total; i0 += PB * DECIDE_THREADS) {
    f4 v[PB];
#pragma unroll
    for (int u = 0; u < PB; ++u) {
      const int i = i0 + u * DECIDE_THREADS;
      if (i < nc * cpr) {
        v[u] = *reinterpret_cast<const f4*>(ctx + (size_t)i * 4);
      } else if (i < total) {
        const int c = (i - nc * cpr) * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[u][e] = to_f<T>(E[c + e]);
      }
    }
#pragma unroll
    for (int u = 0; u < PB; ++u) {
      const int i = i0 + u * DECIDE_THREADS;
      if (i < total) *reinterpret_cast<f4*>(x + (size_t)i * 4) = v[u];
    }
  }
}

// Sum the split-K partials of a GEMM in split order and apply its epilogue.
// SwiGLU: output feature f pairs gate column 16*(f/8) + f%8 with the up column 8 after it.
// Grid (output columns / 256, rows): one output per thread, its partial loads
// (nsplit <= SPLIT_RED_MAX) all in flight before they are added in split order.
constexpr int SPLIT_RED_MAX = 16;
template <typename T, int EPI>
__global__ __launch_bounds__(256) void k_split_reduce(GemmArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  const int m = blockIdx.y;
  const float* pm = a.part + (size_t)m * a.N;
  const size_t ss = (size_t)a.M * a.N;
  const int ns = a.nsplit;
  if constexpr (EPI == EPI_SWIGLU) {
    const int f = blockIdx.x * 256 + threadIdx.x;
    if (f >= a.N / 2) return;
    const int ng = (f / 8) * 16 + f % 8;
    float g[SPLIT_RED_MAX], u[SPLIT_RED_MAX];
#pragma unroll
    for (int s = 0; s < SPLIT_RED_MAX; ++s)
      if (s < ns) {
        g[s] = pm[s * ss + ng];
        u[s] = pm[s * ss + ng + 8];
      }
    float gv = 0.f, uv = 0.f;
#pragma unroll
    for (int s = 0; s < SPLIT_RED_MAX; ++s)
      if (s < ns) {
        gv += g[s];
        uv += u[s];
      }
    Act<T>::put(a.out, m, a.ldo, f, gv / (1.0f + expf(-gv)) * uv);
    return;
  }
  const int n = blockIdx.x * 256 + threadIdx.x;
  if (n >= a.N) return;
  float p[SPLIT_RED_MAX];
#pragma unroll
  for (int s = 0; s < SPLIT_RED_MAX; ++s)
    if (s < ns) p[s] = pm[s * ss + n];
  float v = 0.f;
#pragma unroll
  for (int s = 0; s < SPLIT_RED_MAX; ++s)
    if (s < ns) v += p[s];
  if constexpr (EPI == EPI_OP) {
    Act<T>::put(a.out, m, a.ldo, n, v);
  } else if constexpr (EPI == EPI_XMASK) {
    if (a.rowmask[m]) ((float*)a.out)[(size_t)m * a.ldo + n] = v;
  } else {
    ((float*)a.out)[(size_t)m * a.ldo + n] = v;
  }
}

// ------------------------------------------------------------------------ big
template <typename T, int EPI>
__global__ __launch_bounds__(256) void k_gemm_big(GemmArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  constexpr int EPL = Frag<T>::EPL, KB = Frag<T>::KB;
  constexpr int LDR = 5;  // u4 per LDS row: 4 used + 1 pad against bank conflicts
  constexpr int NA = Act<T>::PL;  // activation planes (hi, lo)
  __shared__ u4 sA[2][NA][128 * LDR];
  __shared__ u4 sB[2][128 * LDR];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int wm = w >> 1, wn = w & 1;
  const int m0 = blockIdx.y * 128, n0 = blockIdx.x * 128;
  const T* W = (const T*)a.W;
  const T* X = (const T*)a.X;
  const int lr = tid >> 1, lc = (tid & 1) * 2;
  const bool aok = m0 + lr < a.M;
  const T* ap = X + (size_t)(aok ? m0 + lr : 0) * a.ldx * NA + lc * EPL;
  // B tile: 8 fragment blocks (16 rows x KB each, 64 u4 in lane order) per stage;
  // thread t copies u4 number 2t and 2t+1 of the 512
  const int nfr = a.K / KB;
  int bidx[2], brow[2], bg[2];
  bool bok[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int u = 2 * tid + q, blk = u >> 6, l = u & 63;
    brow[q] = blk * 16 + (l & 15);
    bg[q] = l >> 4;
    bok[q] = n0 + blk * 16 < a.N;
    bidx[q] = l;
  }
  const int nt0 = n0 / 16;
  const int nst = a.K / KB;
  u4 ra[NA][2], rb[2];
  auto gload = [&](int s) {
    const size_t k = (size_t)s * KB;
#pragma unroll
    for (int p = 0; p < NA; ++p) {
      ra[p][0] = aok ? ld16(ap + (size_t)p * a.ldx + k) : zero16();
      ra[p][1] = aok ? ld16(ap + (size_t)p * a.ldx + k + EPL) : zero16();
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const size_t blk = (size_t)(nt0 + (brow[q] >> 4)) * nfr + s;
      rb[q] = bok[q] ? ld16_stream(W + (blk * 64 + bidx[q]) * EPL) : zero16();
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int p = 0; p < NA; ++p) {
      sA[buf][p][lr * LDR + lc] = ra[p][0];
      sA[buf][p][lr * LDR + lc + 1] = ra[p][1];
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) sB[buf][brow[q] * LDR + bg[q]] = rb[q];
  };
  f4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  gload(0);
  sstore(0);
  __syncthreads();
  for (int s = 0; s < nst; ++s) {
    const int cur = s & 1;
    if (s + 1 < nst) gload(s + 1);
    u4 af[4], afl[4], bfr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      af[i] = sA[cur][0][(wm * 64 + i * 16 + r16) * LDR + g];
      afl[i] = sA[cur][NA - 1][(wm * 64 + i * 16 + r16) * LDR + g];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) bfr[j] = sB[cur][(wn * 64 + j * 16 + r16) * LDR + g];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) mma_act<T>(acc[i][j], af[i], afl[i], bfr[j]);
    if (s + 1 < nst) sstore(cur ^ 1);
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int nb = n0 + wn * 64 + 16 * j;
      if (nb >= a.N) continue;  // uniform per wave
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm * 64 + i * 16 + 4 * g + r;
        epi_tile<T, EPI>(a, m, m < a.M, nb, r16, acc[i][j][r]);
      }
    }
}

// ------------------------------------------------------------------------ prompt GEMM
// Prompt chunks (M > 256 rows): a BM x 128 output tile per workgroup of BM/32
// waves (64 x 64 each), k in steps of one fragment (KB).  Every operand
// fragment a wave reads is one 1 KB block in lane order, and it lands in LDS
// in that order straight from memory (global_load_lds_dwordx4: no registers
// in flight), in a ring of PF_NS stages with PF_NS - 1 stages in flight, so a
// step waits on memory only if the loads of a stage take longer than the
// matrix work of the stages before it.  A fragment of X (16 rows, one k-slice)
// is read by lane l from row l & 15 at k-offset (l >> 4) * EPL; a weight
// fragment is already a contiguous 1 KB block (fragment-tiled layout).
// Rows past M read row M - 1 and tiles past N the last tile (never stored).
#ifndef HAM_PF_NS
#define HAM_PF_NS 3
#endif
constexpr int PF_NS = HAM_PF_NS;

// s_waitcnt with vmcnt <= n (0..63) and lgkmcnt = 0 (expcnt untouched)
template <int N>
__device__ __forceinline__ void wait_vm_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

// Output tile of a prompt-GEMM workgroup.  Workgroups go to the 8 XCDs in
// turn (linear id mod 8), and each XCD has its own L2: the grid is renumbered
// so that every XCD takes one contiguous range of tiles, ordered in groups of
// PF_GM M-tiles (M fastest), so the ~32 workgroups an XCD runs at once share
// their X and weight slices in its L2 (4 M-tiles x 8 N-tiles at a time).
#ifndef HAM_PF_GM
#define HAM_PF_GM 4
#endif
__device__ __forceinline__ void pf_tile(int& mt, int& nt) {
  const int gx = gridDim.x, gy = gridDim.y, G = gx * gy;
  int L = blockIdx.y * gx + blockIdx.x;
  if (HAM_PF_GM == 0) {
    mt = blockIdx.y;
    nt = blockIdx.x;
    return;
  }
  if (G % 8 == 0) L = (L % 8) * (G / 8) + L / 8;
  const int per_group = HAM_PF_GM * gx, group = L / per_group, first_m = group * HAM_PF_GM;
  const int gsz = min(gy - first_m, HAM_PF_GM), r = L - group * per_group;
  mt = first_m + r % gsz;
  nt = r / gsz;
}

template <typename T, int EPI, int BM, int BN>
__global__ __launch_bounds__(BM / 64 * 2 * 64) void k_gemm_pf(GemmArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  constexpr int EPL = Frag<T>::EPL, KB = Frag<T>::KB, PL = Act<T>::PL;
  constexpr int NW = BM / 64 * 2;                // waves: BM/64 rows x 2 columns of 64 x BN/2
  constexpr int WT = BN / 32;                    // 16-column tiles per wave
  constexpr int NA = (BM / 16) * PL, NBW = BN / 16;  // 1 KB fragments per stage: X (tiles x planes), W (tiles)
  constexpr int NL = NA + NBW, LPW = NL / NW;    // wave-loads per stage, per wave
  static_assert(NL % NW == 0, "loads per stage must split evenly over the waves");
  constexpr int FRAG = 64;                       // u4 per fragment
  __shared__ u4 ring[PF_NS][NL * FRAG];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int wm = w >> 1, wn = w & 1;
  int mt, nt;
  pf_tile(mt, nt);
  const int m0 = mt * BM, n0 = nt * BN;
  const int nfr = a.K / KB, ntile = a.N / 16;
  const T* W = (const T*)a.W;
  const T* X = (const T*)a.X;
  // this wave's loads of a stage: fragment q = w + NW * i (X fragments first)
  const T* src[LPW];
  int dst[LPW];
  bool isw[LPW];
#pragma unroll
  for (int i = 0; i < LPW; ++i) {
    const int q = w + NW * i;
    dst[i] = q * FRAG;
    if (q < NA) {
      const int t = q / PL, p = q % PL;
      const int m = min(m0 + t * 16 + r16, a.M - 1);
      src[i] = X + ((size_t)m * PL + p) * a.ldx + g * EPL;
      isw[i] = false;
    } else {
      const int t = min(n0 / 16 + (q - NA), ntile - 1);
      src[i] = W + (size_t)t * nfr * FRAG * EPL + (size_t)lane * EPL;
      isw[i] = true;
    }
  }
  auto issue = [&](int s) {  // stage s (k-fragment s) into ring slot s % PF_NS
    u4* slot = ring[s % PF_NS];
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
      const T* p = src[i] + (size_t)s * (isw[i] ? FRAG * EPL : KB);
      __builtin_amdgcn_global_load_lds((const void*)p, (__attribute__((address_space(3))) void*)(slot + dst[i]), 16,
                                       0, 0);
    }
  };
  f4 acc[4][WT];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < WT; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  const int nst = nfr;
#pragma unroll
  for (int s = 0; s < PF_NS - 1; ++s)
    if (s < nst) issue(s);
  for (int s = 0; s < nst; ++s) {
    // stage s has landed once at most the loads of the stages issued after it are pending
    if (s + PF_NS - 2 < nst) wait_vm_lgkm0<(PF_NS - 2) * LPW>();
    else wait_vm_lgkm0<0>();
    asm volatile("s_barrier" ::: "memory");
    // every wave is past stage s - 1: its slot takes stage s + PF_NS - 1
    if (s + PF_NS - 1 < nst) issue(s + PF_NS - 1);
    const u4* slot = ring[s % PF_NS];
    u4 af[4][PL], bf[WT];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int p = 0; p < PL; ++p) af[i][p] = slot[((wm * 4 + i) * PL + p) * FRAG + lane];
#pragma unroll
    for (int j = 0; j < WT; ++j) bf[j] = slot[(NA + wn * WT + j) * FRAG + lane];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < WT; ++j) mma_act<T>(acc[i][j], af[i][0], af[i][PL - 1], bf[j]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < WT; ++j) {
      const int nb = n0 + wn * (BN / 2) + 16 * j;
      if (nb >= a.N) continue;  // uniform per wave
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm * 64 + i * 16 + 4 * g + r;
        epi_tile<T, EPI>(a, m, m < a.M, nb, r16, acc[i][j][r]);
      }
    }
}

// ------------------------------------------------------------------------ launch
// compute units of the target part (MI355X: 256 in 8 XCDs)
constexpr int GPU_CUS = 256;

// Split-K count for a grid of `ntiles` column tiles: the one whose busiest CU
// streams the least (a count that leaves some CUs one workgroup more than the
// others costs that workgroup's bytes on all of them), and among those the
// grid nearest `target` workgroups; at most `cap`.
static int balanced_split(int ntiles, int cap, int target) {
  cap = std::max(1, cap);
  double best_load = 1e30;
  long best_dist = 1L << 40;
  int best = 1;
  for (int ns = 1; ns <= cap; ++ns) {
    const long wgs = (long)ntiles * ns;
    const double load = (double)((wgs + GPU_CUS - 1) / GPU_CUS) / ns;
    const long dist = std::labs(wgs - target);
    if (load < best_load * (1 - 1e-9) || (load <= best_load * (1 + 1e-9) && dist < best_dist)) {
      best_load = std::min(best_load, load);
      best_dist = dist;
      best = ns;
    }
  }
  return best;
}

// column tiles of a skinny launch: 32-column tiles while they already give
// enough workgroups, else 16-column tiles
int skinny_tiles(int N) { return (N / 32 >= 512) ? N / 32 : N / 16; }

template <typename T, int MT, int TN, int EPI>
static void run_skinny(const GemmArgs& a, int nsplit, int tag, Stream s) {
  dim3 grid(a.N / (16 * TN), nsplit);
  if constexpr (EPI == EPI_F32 || EPI == EPI_RESID || EPI == EPI_SWIGLU) {
    if (!tag) {
      launch_k((k_gemm_skinny<T, MT, TN, EPI, 0>), grid, dim3(256), 0, s, a);
      return;
    }
  }
  launch_k((k_gemm_skinny<T, MT, TN, EPI, 1>), grid, dim3(256), 0, s, a);
}

// 16-column tiles only (at 32 columns the 16-wave kernel spills registers)
int gemm_norm_out_tiles(int N) {
  if (N % 32 != 0 || N / 16 > NORM_OUT_MAX_TILES) return -1;
  return N / 16;
}

bool gemm_norm_out_fits(int M, int N, int K) {
  return M >= 1 && M <= NORM_OUT_MAX_ROWS && K > 0 && gemm_norm_out_tiles(N) > 0;
}

// NormOut launch: one workgroup of 16 waves per column tile over the whole k-range
template <typename T>
static int run_norm_out(const GemmArgs& a, int tag, Stream s) {
  if (!gemm_norm_out_fits(a.M, a.N, a.K) || a.K % Frag<T>::KB || !a.no.ss || (a.no.g && !a.no.act)) return -1;
  const dim3 grid(gemm_norm_out_tiles(a.N)), block(64 * 16);
  if (!tag) launch_k((k_gemm_skinny<T, 1, 1, EPI_RESID, 0, 16>), grid, block, 0, s, a);
  else launch_k((k_gemm_skinny<T, 1, 1, EPI_RESID, 1, 16>), grid, block, 0, s, a);
  return 0;
}

template <typename T, int TN, int EPI>
static void run_skinny_mt(const GemmArgs& a, int nsplit, int tag, Stream s) {
  const int mt = (a.M + 15) / 16;
  if (mt == 1) run_skinny<T, 1, TN, EPI>(a, nsplit, tag, s);
  else if (mt == 2) run_skinny<T, 2, TN, EPI>(a, nsplit, tag, s);
  else run_skinny<T, 4, TN, EPI>(a, nsplit, tag, s);
}

template <typename T, int TN, int EPI, int XS>
static void run_staged(const GemmArgs& a, int nsplit, int tag, size_t lds, Stream s) {
  dim3 grid(a.N / (16 * TN), nsplit);
  if (!tag) launch_k((k_gemm_staged<T, TN, EPI, 0, XS>), grid, dim3(STG_THREADS), lds, s, a);
  else launch_k((k_gemm_staged<T, TN, EPI, 1, XS>), grid, dim3(STG_THREADS), lds, s, a);
}

// Staged launch (X built in LDS): k-split and the checks that the prologue fits.
// Returns GEMM_NO_STAGE if it does not; launches unless dry.
template <typename T, int EPI>
static int gemm_staged(const GemmArgs& a0, int max_split, int tag, Stream s, int* nsplit_out, bool dry) {
  constexpr int KB = Frag<T>::KB;
  GemmArgs a = a0;
  constexpr bool norm_ok = EPI == EPI_F32 || EPI == EPI_SWIGLU;
  constexpr bool attn_ok = EPI == EPI_RESID;
  if ((a.xsrc == XS_NORM && !norm_ok) || (a.xsrc == XS_ATTN && !attn_ok)) return GEMM_NO_STAGE;
  if (a.M > STG_MMAX) return GEMM_NO_STAGE;
  const int nfr = a.K / KB;
  const int ntiles = skinny_tiles(a.N);
  const int TN = a.N / (16 * ntiles);
  int nsplit = 1;
  if (EPI != EPI_SWIGLU && max_split > 1) {
    // at most about 512 workgroups (two per CU fit at once), two fragments per
    // wave; not balanced per CU as the plain path is: every workgroup repeats
    // the prologue, which a larger grid pays for more than it gains
    nsplit = std::max(1, 512 / ntiles);
    nsplit = std::max(1, std::min(nsplit, std::min(max_split, nfr / (2 * STG_NW))));
  }
  const int Kr = (nfr + nsplit - 1) / nsplit * KB;  // longest k-range
  if (a.M * Kr > STG_VALS) return GEMM_NO_STAGE;
  if (a.xsrc == XS_NORM) {
    if (a.xs.part && (a.xs.nsplit < 1 || a.xs.nsplit > STG_SMAX)) return GEMM_NO_STAGE;
    if (nsplit > 1 && !a.xs.ss_out) return GEMM_NO_STAGE;
  } else {
    // every workgroup reads the attention records of its k-range: only while
    // there are few of them (a thread combines at most STG_AMAX splits)
    const int nch = a.M * Kr / 4, ans = a.xs.ans;
    if (nch > STG_THREADS || ans > 64) return GEMM_NO_STAGE;
    const int SG = std::max(1, std::min(STG_THREADS / nch, ans));
    if ((ans + SG - 1) / SG > STG_AMAX) return GEMM_NO_STAGE;
  }
  const size_t lds = stage_lds_bytes(TN, a.M, Kr, a.xsrc, a.xs.ans, a.xs.hd);
  if (lds > 64 * 1024) return GEMM_NO_STAGE;
  *nsplit_out = nsplit;
  if (dry) return 0;
  a.nsplit = nsplit;
  if constexpr (norm_ok) {
    if (TN == 2) run_staged<T, 2, EPI, XS_NORM>(a, nsplit, tag, lds, s);
    else run_staged<T, 1, EPI, XS_NORM>(a, nsplit, tag, lds, s);
  } else if constexpr (attn_ok) {
    if (TN == 2) run_staged<T, 2, EPI, XS_ATTN>(a, nsplit, tag, lds, s);
    else run_staged<T, 1, EPI, XS_ATTN>(a, nsplit, tag, lds, s);
  }
  return 0;
}

// Batched rows: X through LDS once per workgroup of eight tiles; about 512
// workgroups, split-K (SwiGLU then finishes in k_split_reduce; the argmax never splits).
template <typename T, int EPI, bool NX = false>
static int gemm_wide(GemmArgs a, int max_split, int tag, Stream s, int* nsplit_out) {
  const int ntiles = skinny_tiles(a.N);
  const int TN = a.N / (16 * ntiles);

    const int groups = (ntiles + WIDE_NW - 1) / WIDE_NW;
    const int nch = a.K / WIDE_KC;
    int nsplit = 1;
    if (EPI != EPI_ARGMAX && (max_split > 1 || EPI == EPI_SWIGLU))
      nsplit = std::max(1, std::min(std::min((512 + groups - 1) / groups, nch),
                                    EPI == EPI_SWIGLU ? MAX_WIDE_SWIGLU_SPLIT : max_split));
    nsplit = std::max(1, std::min(nsplit, PART_ROWS / a.M));
    a.nsplit = nsplit;
    *nsplit_out = EPI == EPI_SWIGLU ? 1 : nsplit;  // SwiGLU partials are finished here
    dim3 grid(groups, nsplit);
    const int mt = (a.M + 15) / 16;
#define HAM_WIDE(MTV, TNV)                                                                              \
    do {                                                                                                \
      if (!tag && (EPI == EPI_F32 || EPI == EPI_RESID || EPI == EPI_SWIGLU))                            \
        launch_k((k_gemm_wide<T, MTV, TNV, EPI, 0, NX>), grid, dim3(64 * WIDE_NW), 0, s, a);            \
      else                                                                                              \
        launch_k((k_gemm_wide<T, MTV, TNV, EPI, 1, NX>), grid, dim3(64 * WIDE_NW), 0, s, a);            \
    } while (0)
    if (TN == 2) {
      if (mt <= 2) HAM_WIDE(2, 2); else if (mt <= 4) HAM_WIDE(4, 2); else if (mt <= 8) HAM_WIDE(8, 2);
      else if (mt <= 10) HAM_WIDE(10, 2); else HAM_WIDE(16, 2);
    } else {
      if (mt <= 2) HAM_WIDE(2, 1); else if (mt <= 4) HAM_WIDE(4, 1); else if (mt <= 8) HAM_WIDE(8, 1);
      else if (mt <= 10) HAM_WIDE(10, 1); else HAM_WIDE(16, 1);
    }
#undef HAM_WIDE
    if (EPI == EPI_SWIGLU && nsplit > 1)
      launch_k((k_split_reduce<T, EPI_SWIGLU>), dim3((a.N / 2 + 255) / 256, a.M), dim3(256), 0, s, a);
    return 0;
  }

template <typename T, int EPI>
static int gemm_t(const GemmArgs& a0, int max_split, int tag, Stream s, int* nsplit_out, bool dry = false) {
  GemmArgs a = a0;
  constexpr int KB = Frag<T>::KB;
  if (a.N % 32 != 0 || a.K % KB != 0 || a.M <= 0) return -1;
  if ((a.no.ss || a.rs.ss) && a.xsrc != XS_ACT) return -1;  // NormOut, RowScale: plain operand only
  *nsplit_out = 1;
  if (a.xsrc == XS_NORMW) {  // normed X built by the batched GEMM itself (8 < M <= 256)
    if constexpr (EPI == EPI_F32 || EPI == EPI_SWIGLU) {
      if (a.M > 8 && a.M <= 256 && a.K % WIDE_KC == 0 && a.xs.x && a.xs.g && a.xs.ssw &&
          a.xs.nchw == (a.K + 255) / 256) {
        if (dry) return 0;
        return gemm_wide<T, EPI, true>(a, max_split, tag, s, nsplit_out);
      }
    }
    return GEMM_NO_STAGE;
  }
  if (a.xsrc != XS_ACT) {
    if constexpr (EPI == EPI_F32 || EPI == EPI_SWIGLU || EPI == EPI_RESID)
      return gemm_staged<T, EPI>(a, max_split, tag, s, nsplit_out, dry);
    else
      return GEMM_NO_STAGE;
  }
  if (dry) return GEMM_NO_STAGE;
  if constexpr (EPI == EPI_RESID) {
    if (a.no.ss) {
      *nsplit_out = 1;
      return run_norm_out<T>(a, tag, s);
    }
  }
  if constexpr (EPI == EPI_SWIGLU) {
    // the row scale is applied by the skinny kernel of one 16-row tile only
    if (a.rs.ss && (a.M > NORM_OUT_MAX_ROWS || a.rs.n < 1 || a.rs.n > NORM_OUT_MAX_TILES)) return -1;
  }
  if (a.M > 8 && a.M <= 256 && a.K % WIDE_KC == 0 && EPI != EPI_XMASK && EPI != EPI_OP)
    return gemm_wide<T, EPI>(a, max_split, tag, s, nsplit_out);
  if (a.M > 64) {
    if constexpr (EPI == EPI_ARGMAX) {
      return -1;
    } else {
#ifndef HAM_PF_BN
#define HAM_PF_BN 256
#endif
      if (a.M > 256) {
        constexpr int BM = 128;
        // 256-column tiles (64 x 128 per wave: half the operand reads from LDS per
        // product of 64 x 64) while they still give at least two workgroups per CU
        if (HAM_PF_BN == 256 && (long)((a.N + 255) / 256) * ((a.M + BM - 1) / BM) >= 512) {
          dim3 grid((a.N + 255) / 256, (a.M + BM - 1) / BM);
          launch_k((k_gemm_pf<T, EPI, BM, 256>), grid, dim3(BM / 64 * 2 * 64), 0, s, a);
        } else {
          dim3 grid((a.N + 127) / 128, (a.M + BM - 1) / BM);
          launch_k((k_gemm_pf<T, EPI, BM, 128>), grid, dim3(BM / 64 * 2 * 64), 0, s, a);
        }
        return 0;
      }
      dim3 grid((a.N + 127) / 128, (a.M + 127) / 128);
      launch_k((k_gemm_big<T, EPI>), grid, dim3(256), 0, s, a);
      return 0;
    }
  }
  const int nfr = a.K / KB;
  const int ntiles = skinny_tiles(a.N);
  const int TN = a.N / (16 * ntiles);
  int nsplit = 1;
  if (EPI != EPI_ARGMAX && EPI != EPI_SWIGLU && max_split > 1) {
    // about 1024 workgroups, at least four fragments per wave
#ifndef HAM_SKINNY_WGS
#define HAM_SKINNY_WGS 1024
#endif
    nsplit = balanced_split(ntiles, std::min(max_split, nfr / 16), HAM_SKINNY_WGS);
  }
  a.nsplit = nsplit;
  *nsplit_out = nsplit;
  if (TN == 2) run_skinny_mt<T, 2, EPI>(a, nsplit, tag, s);
  else run_skinny_mt<T, 1, EPI>(a, nsplit, tag, s);
  return 0;
}

template <typename T>
static int gemm_dispatch(int epi, const GemmArgs& a, int max_split, int tag, Stream s, int* ns, bool dry) {
  switch (epi) {
    case EPI_F32: return gemm_t<T, EPI_F32>(a, max_split, tag, s, ns, dry);
    case EPI_OP: return gemm_t<T, EPI_OP>(a, max_split, tag, s, ns, dry);
    case EPI_RESID: return gemm_t<T, EPI_RESID>(a, max_split, tag, s, ns, dry);
    case EPI_SWIGLU: return gemm_t<T, EPI_SWIGLU>(a, max_split, tag, s, ns, dry);
    case EPI_ARGMAX: return gemm_t<T, EPI_ARGMAX>(a, max_split, tag, s, ns, dry);
    case EPI_XMASK: return gemm_t<T, EPI_XMASK>(a, max_split, tag, s, ns, dry);
  }
  return -1;
}

int launch_gemm(int dtype, int epi, const GemmArgs& a, int max_split, Stream s, int tag, int* nsplit) {
  int ns = 1;
  const int rc = dtype == 1 ? gemm_dispatch<bf16>(epi, a, max_split, tag, s, &ns, false)
                            : gemm_dispatch<float>(epi, a, max_split, tag, s, &ns, false);
  if (nsplit) *nsplit = ns;
  return rc;
}

bool gemm_stage_fits(int dtype, int epi, const GemmArgs& a, int max_split) {
  int ns = 1;
  const int rc = dtype == 1 ? gemm_dispatch<bf16>(epi, a, max_split, 1, nullptr, &ns, true)
                            : gemm_dispatch<float>(epi, a, max_split, 1, nullptr, &ns, true);
  return rc == 0;
}

int launch_decide(int dtype, const DecideArgs& d, int ntiles, int M, Stream s) {
  // ntiles: argmax partials written per row by the LM-head launch
  if (ntiles > DECIDE_THREADS * DECIDE_PER || ntiles != d.ntiles) return -1;
  if (d.prep_k < 0 || d.prep_k > 3) return -1;
  if (dtype == 1) launch_k(k_decide<bf16>, dim3(M), dim3(DECIDE_THREADS), 0, s, d, ntiles);
  else launch_k(k_decide<float>, dim3(M), dim3(DECIDE_THREADS), 0, s, d, ntiles);
  return 0;
}

int launch_split_reduce(int dtype, int epi, const GemmArgs& a, Stream s) {
  if (a.nsplit < 1 || a.nsplit > SPLIT_RED_MAX) return -1;
  dim3 grid((a.N + 255) / 256, a.M);
#define HAM_RED(EP)                                                                                     \
  do {                                                                                                  \
    if (dtype == 1) launch_k((k_split_reduce<bf16, EP>), grid, dim3(256), 0, s, a);           \
    else launch_k((k_split_reduce<float, EP>), grid, dim3(256), 0, s, a);                    \
  } while (0)
  if (epi == EPI_OP) HAM_RED(EPI_OP);
  else if (epi == EPI_XMASK) HAM_RED(EPI_XMASK);
  else if (epi == EPI_F32) HAM_RED(EPI_F32);
  else if (epi == EPI_SWIGLU) HAM_RED(EPI_SWIGLU);
  else return -1;
#undef HAM_RED
  return 0;
}

}  // namespace ham
