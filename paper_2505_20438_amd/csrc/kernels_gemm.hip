// Weight GEMMs of the decode loop: C[m][n] = sum_k X[m][k] * W[n][k].
//
// Two matrix-core kernels share one set of fused epilogues:
//  * k_gemm_skinny (M <= 64 rows: decode, micro steps, LM head).  HBM-bound
//    weight streaming: each lane loads 16 contiguous bytes of a weight row per
//    fragment (non-temporal), four waves split the k-range of a 16*TN-column
//    tile, and the k dimension may additionally be split across workgroups,
//    reduced in a fixed order by the last workgroup to finish (deterministic,
//    no spinning).  X rows are the A operand (padded to 16), weight rows the B
//    operand, so the accumulator's columns are output features.
//  * k_gemm_big (M > 64: prefill chunks, batched micro context rows): 128x128
//    LDS-staged tiles, double buffered, 2x2 waves of 64x64.
#include "decide.h"
#include "device_common.h"
#include "ham_internal.h"

namespace ham {

template <typename T, int EPI>
__device__ __forceinline__ void epi_pair(const GemmArgs& a, int m, int nb, int r16, float ve, float vo) {
  const int ne = nb + r16, no = nb + 16 + r16;
  if constexpr (EPI == EPI_F32) {
    float* o = (float*)a.out + (size_t)m * a.ldo;
    o[ne] = ve;
    o[no] = vo;
  } else if constexpr (EPI == EPI_OP) {
    Act<T>::put(a.out, m, a.ldo, ne, ve);
    Act<T>::put(a.out, m, a.ldo, no, vo);
  } else if constexpr (EPI == EPI_RESID) {
    float* o = (float*)a.out + (size_t)m * a.ldo;
    const float xe = o[ne] + ve, xo = o[no] + vo;
    o[ne] = xe;
    o[no] = xo;
    if (a.ctx) {
      a.ctx[(size_t)m * a.ldctx + ne] = xe;
      a.ctx[(size_t)m * a.ldctx + no] = xo;
    }
  } else if constexpr (EPI == EPI_XMASK) {
    if (a.rowmask[m]) {
      float* o = (float*)a.out + (size_t)m * a.ldo;
      o[ne] = ve;
      o[no] = vo;
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    // gate rows and up rows are interleaved in blocks of 16: pair (gate, up) of feature f
    const float sg = ve / (1.0f + expf(-ve));
    Act<T>::put(a.out, m, a.ldo, nb / 2 + r16, sg * vo);
  }
}

__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

// ------------------------------------------------------------------------ skinny
template <typename T, int TN, int MT, int EPI>
__global__ __launch_bounds__(256) void k_gemm_skinny(GemmArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  constexpr int EPL = Frag<T>::EPL, KB = Frag<T>::KB;
  constexpr int NACC = MT * TN * 4;
  __shared__ float red[3][NACC][64];
  __shared__ int sh_flag;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int ntile = blockIdx.x, split = blockIdx.y, nsplit = gridDim.y;
  const int n0 = ntile * 16 * TN;
  const int nfr = a.K / KB;
  const int c0 = (int)((long)split * nfr / nsplit), c1 = (int)((long)(split + 1) * nfr / nsplit);
  const int f0 = c0 + w * (c1 - c0) / 4, f1 = c0 + (w + 1) * (c1 - c0) / 4;
  const T* W = (const T*)a.W;
  const T* X = (const T*)a.X;

  f4 acc[MT][TN];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  const T* wrow[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) wrow[j] = W + (size_t)(n0 + 16 * j + r16) * a.K + g * EPL;
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

  constexpr int U = 4;
  int f = f0;
  for (; f + U <= f1; f += U) {
    u4 bw[U][TN];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < TN; ++j) bw[u][j] = ld16_stream(wrow[j] + (size_t)(f + u) * KB);
    u4 ax[U][MT], axl[U][MT];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        ax[u][i] = xok[i] ? ld16(xrow[i] + (size_t)(f + u) * KB) : zero16();
        axl[u][i] = (Act<T>::SPLIT && xok[i]) ? ld16(xrow[i] + lo_off + (size_t)(f + u) * KB) : zero16();
      }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) mma_act<T>(acc[i][j], ax[u][i], axl[u][i], bw[u][j]);
  }
  for (; f < f1; ++f) {
    u4 bw[TN], ax[MT], axl[MT];
#pragma unroll
    for (int j = 0; j < TN; ++j) bw[j] = ld16_stream(wrow[j] + (size_t)f * KB);
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      ax[i] = xok[i] ? ld16(xrow[i] + (size_t)f * KB) : zero16();
      axl[i] = (Act<T>::SPLIT && xok[i]) ? ld16(xrow[i] + lo_off + (size_t)f * KB) : zero16();
    }
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) mma_act<T>(acc[i][j], ax[i], axl[i], bw[j]);
  }

  // reduce the four waves' k-slices (fixed order: wave 0 + 1 + 2 + 3)
  if (w > 0) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[w - 1][(i * TN + j) * 4 + r][lane] = acc[i][j][r];
  }
  __syncthreads();
  if (w == 0) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int q = (i * TN + j) * 4 + r;
          acc[i][j][r] = ((acc[i][j][r] + red[0][q][lane]) + red[1][q][lane]) + red[2][q][lane];
        }
  }

  if (nsplit > 1) {
    // publish this k-chunk; the last workgroup of the column tile reduces all chunks in order
    if (w == 0) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int m = 16 * i + 4 * g + r;
            if (m < a.M) a.part[((size_t)split * a.M + m) * a.N + n0 + 16 * j + r16] = acc[i][j][r];
          }
    }
    if (!last_arriver(a.counters + ntile, nsplit, &sh_flag)) return;
    if (w == 0) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int m = 16 * i + 4 * g + r;
            float s = 0.f;
            if (m < a.M)
              for (int c = 0; c < nsplit; ++c) s += a.part[((size_t)c * a.M + m) * a.N + n0 + 16 * j + r16];
            acc[i][j][r] = s;
          }
    }
  }

  if constexpr (EPI == EPI_ARGMAX) {
    const DecideArgs& d = a.dec;
    if (w == 0) {
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
            d.best_val[(size_t)ntile * a.M + m] = bv;
            d.best_idx[(size_t)ntile * a.M + m] = bi;
          }
        }
    }
    if (!last_arriver(a.counters + gridDim.x, gridDim.x, &sh_flag)) return;
    // final argmax per row over all workgroups, then the decision
    for (int m = w; m < a.M; m += 4) {
      float bv = -INFINITY;
      int bi = 0x7fffffff;
      for (int t = lane; t < (int)gridDim.x; t += 64) {
        const float v = d.best_val[(size_t)t * a.M + m];
        const int i = d.best_idx[(size_t)t * a.M + m];
        if (better(v, i, bv, bi)) { bv = v; bi = i; }
      }
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const float ov = __shfl_xor(bv, o, WAVE);
        const int oi = __shfl_xor(bi, o, WAVE);
        if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
      }
      if (lane == 0) decide_one(d, m, bi, d.stop_buf[m]);
    }
  } else {
    if (w == 0) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < TN; j += 2)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int m = 16 * i + 4 * g + r;
            if (m < a.M) epi_pair<T, EPI>(a, m, n0 + 16 * j, r16, acc[i][j][r], acc[i][j + 1][r]);
          }
    }
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
  const bool aok = m0 + lr < a.M, bok = n0 + lr < a.N;
  const T* ap = X + (size_t)(aok ? m0 + lr : 0) * a.ldx * NA + lc * EPL;
  const T* bp = W + (size_t)(bok ? n0 + lr : 0) * a.K + lc * EPL;
  const int nst = a.K / KB;
  u4 ra[NA][2], rb0, rb1;
  auto gload = [&](int s) {
    const size_t k = (size_t)s * KB;
#pragma unroll
    for (int p = 0; p < NA; ++p) {
      ra[p][0] = aok ? ld16(ap + (size_t)p * a.ldx + k) : zero16();
      ra[p][1] = aok ? ld16(ap + (size_t)p * a.ldx + k + EPL) : zero16();
    }
    rb0 = bok ? ld16_stream(bp + k) : zero16();
    rb1 = bok ? ld16_stream(bp + k + EPL) : zero16();
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int p = 0; p < NA; ++p) {
      sA[buf][p][lr * LDR + lc] = ra[p][0];
      sA[buf][p][lr * LDR + lc + 1] = ra[p][1];
    }
    sB[buf][lr * LDR + lc] = rb0;
    sB[buf][lr * LDR + lc + 1] = rb1;
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
    for (int p = 0; p < 2; ++p) {
      const int nb = n0 + wn * 64 + 32 * p;
      if (nb >= a.N) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm * 64 + i * 16 + 4 * g + r;
        if (m < a.M) epi_pair<T, EPI>(a, m, nb, r16, acc[i][2 * p][r], acc[i][2 * p + 1][r]);
      }
    }
}

// ------------------------------------------------------------------------ launch
template <typename T, int TN, int MT, int EPI>
static void run_skinny(const GemmArgs& a, int nsplit, Stream s) {
  dim3 grid(a.N / (16 * TN), nsplit);
  hipLaunchKernelGGL((k_gemm_skinny<T, TN, MT, EPI>), grid, dim3(256), 0, s, a);
}

template <typename T, int EPI>
static int gemm_t(const GemmArgs& a0, int max_split, Stream s) {
  GemmArgs a = a0;
  constexpr int KB = Frag<T>::KB;
  if (a.N % 32 != 0 || a.K % KB != 0 || a.M <= 0) return -1;
  if (a.M > 64) {
    if constexpr (EPI == EPI_ARGMAX) {
      return -1;
    } else {
      dim3 grid((a.N + 127) / 128, (a.M + 127) / 128);
      hipLaunchKernelGGL((k_gemm_big<T, EPI>), grid, dim3(256), 0, s, a);
      return 0;
    }
  }
  constexpr int TN = 2;
  const int ntiles = a.N / (16 * TN);
  const int nfr = a.K / KB;
  int nsplit = 1;
  if (EPI != EPI_ARGMAX) {
    const int target = 1024;
    nsplit = (target + ntiles - 1) / ntiles;
    if (nsplit > max_split) nsplit = max_split;
    if (nsplit > nfr / 4) nsplit = nfr / 4;
    if (nsplit < 1) nsplit = 1;
  }
  a.nsplit = nsplit;
  const int mt = (a.M + 15) / 16;
  if (mt == 1) run_skinny<T, TN, 1, EPI>(a, nsplit, s);
  else if (mt == 2) run_skinny<T, TN, 2, EPI>(a, nsplit, s);
  else run_skinny<T, TN, 4, EPI>(a, nsplit, s);
  return 0;
}

template <typename T>
static int gemm_dispatch(int epi, const GemmArgs& a, int max_split, Stream s) {
  switch (epi) {
    case EPI_F32: return gemm_t<T, EPI_F32>(a, max_split, s);
    case EPI_OP: return gemm_t<T, EPI_OP>(a, max_split, s);
    case EPI_RESID: return gemm_t<T, EPI_RESID>(a, max_split, s);
    case EPI_SWIGLU: return gemm_t<T, EPI_SWIGLU>(a, max_split, s);
    case EPI_ARGMAX: return gemm_t<T, EPI_ARGMAX>(a, max_split, s);
    case EPI_XMASK: return gemm_t<T, EPI_XMASK>(a, max_split, s);
  }
  return -1;
}

int launch_gemm(int dtype, int epi, const GemmArgs& a, int max_split, Stream s) {
  return dtype == 1 ? gemm_dispatch<bf16>(epi, a, max_split, s) : gemm_dispatch<float>(epi, a, max_split, s);
}

}  // namespace ham
