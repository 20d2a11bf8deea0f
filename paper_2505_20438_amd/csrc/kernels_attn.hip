// Attention over the smashed KV cache (one slot per fused group, Sec. 3.1).
//
// Cache layout per layer: K [seq][kv_head][slot][hd] and V stored d-major,
// VT [seq][kv_head][hd][slot], so that both products are matrix-core
// contractions fed by 16-byte contiguous loads:
//   S^T = K Q^T   (A = K rows, B = Q^T)  and  O = P V  (A = P, B = VT rows).
// The rows of the K operand are permuted so that the score tile lands in the
// registers exactly where the P operand of the next product needs it (lane
// l holds the probabilities of row l & 15 for the slot slice of lane group
// l >> 4), so no data moves between the two products.
//
// k_attn_decode: one workgroup per (query row, kv head, slot split), its waves
//   sharing the slot range.  The rows of the matrix products are the q-heads
//   sharing the kv head (GQA).  Waves merge in LDS; splits (long contexts only)
//   write (max, sum, unnormalised output) and k_attn_combine merges them with
//   the log-sum-exp rule in split order.  Used for base decode (ragged kv_len per sequence) and the micro
//   decoder's local cache.
// k_attn_prefill: four waves of 16 consecutive query rows of one head, causal.
//
// Softmax statistics are fp32.  For bf16 caches the probabilities enter the
// bf16 product as a hi + lo pair (about 16 significant bits).
#include "device_common.h"
#include "ham_internal.h"
#include "rows.h"

namespace ham {

template <typename T> struct PFrag;
template <> struct PFrag<bf16> {
  // probabilities of one lane (8 slots) -> A-operand fragments (hi, lo)
  static __device__ __forceinline__ void make(const float* p, u4& hi, u4& lo) {
    float r[8];
    hi = pack_frag_bf16(p);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t w = (e & 1) ? (hi[e >> 1] >> 16) : (hi[e >> 1] & 0xFFFFu);
      r[e] = p[e] - bf2f((bf16)w);
    }
    lo = pack_frag_bf16(r);
  }
  static constexpr bool TWO = true;
};
template <> struct PFrag<float> {
  static __device__ __forceinline__ void make(const float* p, u4& hi, u4& lo) {
    hi = u4{__float_as_uint(p[0]), __float_as_uint(p[1]), __float_as_uint(p[2]), __float_as_uint(p[3])};
    lo = hi;
  }
  static constexpr bool TWO = false;
};

// The K and V fragments of one key block of KB slots, loaded together (V does
// not depend on the scores, so both streams are in flight at once).
template <typename T, int HD>
struct KVBlock {
  static constexpr int KB = Frag<T>::KB, NF = HD / KB, ND = HD / 16, TT = KB / 16;
  u4 k[TT][NF];
  u4 v[ND];
};

template <typename T, int HD>
__device__ __forceinline__ void kv_load(KVBlock<T, HD>& blk, const T* Kb, const T* Vb, int S, int base) {
  using B = KVBlock<T, HD>;
  constexpr int EPL = Frag<T>::EPL, KB = B::KB;
  const int lane = threadIdx.x & 63, r16 = lane & 15, g = lane >> 4;
#pragma unroll
  for (int t = 0; t < B::TT; ++t) {
    // operand row r16 of tile t holds the slot whose score lane group r16/4 needs
    const int slot = base + (r16 >> 2) * (KB / 4) + 4 * t + (r16 & 3);
    const T* kp = Kb + (size_t)slot * HD + g * EPL;
#pragma unroll
    for (int f = 0; f < B::NF; ++f) blk.k[t][f] = ld16_stream(kp + f * KB);
  }
  const T* vp = Vb + (size_t)r16 * S + base + g * (KB / 4);
#pragma unroll
  for (int dt = 0; dt < B::ND; ++dt) blk.v[dt] = ld16_stream(vp + (size_t)dt * 16 * S);
}

// Scores of the 16 operand rows against the block (lane: row r16, slots
// base + g*KB/4 + e), masked at `limit`, then the online-softmax update of
// (m, l, o) and the P.V product.
template <typename T, int HD>
__device__ __forceinline__ void attn_block(const KVBlock<T, HD>& blk, int base, int limit, const u4* qf,
                                           const u4* ql, float scale, float& mrun, float& lrun, f4* o) {
  using B = KVBlock<T, HD>;
  constexpr int KB = B::KB, ND = B::ND, TT = B::TT;
  const int lane = threadIdx.x & 63, g = lane >> 4;
  float sc[KB / 4];
#pragma unroll
  for (int t = 0; t < TT; ++t) {
    f4 s = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int f = 0; f < B::NF; ++f) mma_act_b<T>(s, blk.k[t][f], qf[f], ql[f]);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int sl = base + g * (KB / 4) + 4 * t + i;
      sc[4 * t + i] = sl < limit ? s[i] * scale : -INFINITY;
    }
  }
  float bm = sc[0];
#pragma unroll
  for (int e = 1; e < KB / 4; ++e) bm = fmaxf(bm, sc[e]);
  bm = fmaxf(bm, __shfl_xor(bm, 16, WAVE));
  bm = fmaxf(bm, __shfl_xor(bm, 32, WAVE));
  const float mnew = fmaxf(mrun, bm);
  const float alpha = (mrun == -INFINITY) ? 0.f : __expf(mrun - mnew);
  float p[KB / 4];
  float ps = 0.f;
#pragma unroll
  for (int e = 0; e < KB / 4; ++e) {
    p[e] = (sc[e] == -INFINITY) ? 0.f : __expf(sc[e] - mnew);
    ps += p[e];
  }
  ps += __shfl_xor(ps, 16, WAVE);
  ps += __shfl_xor(ps, 32, WAVE);
  lrun = lrun * alpha + ps;
  mrun = mnew;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float ai = __shfl(alpha, 4 * g + i, WAVE);
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) o[dt][i] *= ai;
  }
  u4 phi, plo;
  PFrag<T>::make(p, phi, plo);
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) {
    Frag<T>::mma(o[dt], phi, blk.v[dt]);
    if constexpr (PFrag<T>::TWO) Frag<T>::mma(o[dt], plo, blk.v[dt]);
  }
}

// blocks [b0, b1) of KB slots from s0, limit `limit`; block i+1 loads while i computes
template <typename T, int HD>
__device__ __forceinline__ void attn_range(const T* Kb, const T* Vb, int S, int s0, int b0, int b1, int limit,
                                           const u4* qf, const u4* ql, float scale, float& mrun, float& lrun,
                                           f4* o) {
  constexpr int KB = Frag<T>::KB;
  if (b0 >= b1) return;
  KVBlock<T, HD> cur, nxt;
  kv_load<T, HD>(cur, Kb, Vb, S, s0 + b0 * KB);
  for (int bk = b0; bk < b1; ++bk) {
    const bool more = bk + 1 < b1;
    if (more) kv_load<T, HD>(nxt, Kb, Vb, S, s0 + (bk + 1) * KB);
    attn_block<T, HD>(cur, s0 + bk * KB, limit, qf, ql, scale, mrun, lrun, o);
    if (more) cur = nxt;
  }
}

// One workgroup per (query row, kv head, slot split); its NW waves take
// consecutive key blocks of the split's slot range and merge their (max, sum,
// output) through LDS in wave order.  With one split the workgroup writes the
// final output; otherwise it writes the split's partial for k_attn_combine.
constexpr int ATTN_NW = 8;

template <typename T, int HD>
__global__ __launch_bounds__(64 * ATTN_NW) void k_attn_decode(AttnArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  constexpr int EPL = Frag<T>::EPL, KB = Frag<T>::KB, NF = HD / KB, ND = HD / 16;
  __shared__ float sO[ATTN_NW][4][HD];   // per wave: output rows of up to 4 q-heads (grp <= 4 here)
  __shared__ float sM[ATTN_NW][16], sL[ATTN_NW][16];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, r16 = lane & 15, g = lane >> 4;
  const int split = blockIdx.x, kvh = blockIdx.y, r = blockIdx.z;
  const int grp = a.H / a.Hkv;
  const RowInfo ri = row_info(a.rm, r);
  const int nval = ri.enabled ? ri.n_valid : 0;
  int chunk = (nval + a.nsplit - 1) / a.nsplit;
  chunk = (chunk + KB - 1) / KB * KB;
  const int s0 = split * chunk;
  const int s1 = min(nval, s0 + chunk);
  // this wave's key blocks: a contiguous share of the split's blocks
  const int nblk = s1 > s0 ? (s1 - s0 + KB - 1) / KB : 0;
  const int b0 = w * nblk / ATTN_NW, b1 = (w + 1) * nblk / ATTN_NW;
  const T* Kb = (const T*)a.K + ri.b * a.sb + kvh * a.sh;
  const T* Vb = (const T*)a.VT + ri.b * a.sb + kvh * a.sh;
  u4 qf[NF], ql[NF];
  constexpr int PL = Act<T>::PL;
  const T* qp = (const T*)a.q + (size_t)r * a.ldq * PL + (size_t)(kvh * grp + r16) * HD + g * EPL;
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    qf[f] = (r16 < grp) ? ld16(qp + f * KB) : zero16();
    ql[f] = (Act<T>::SPLIT && r16 < grp) ? ld16(qp + a.ldq + f * KB) : zero16();
  }
  f4 o[ND];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) o[dt] = f4{0.f, 0.f, 0.f, 0.f};
  float mrun = -INFINITY, lrun = 0.f;
  const float scale = 1.0f / sqrtf((float)HD);
  attn_range<T, HD>(Kb, Vb, a.S, s0, b0, b1, s1, qf, ql, scale, mrun, lrun, o);

  // publish this wave's state; rows 4g+i of the output live in lane group g
  if (g == 0) {
    sM[w][r16] = mrun;
    sL[w][r16] = lrun;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int j = 4 * g + i;
    if (j < grp) {
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) sO[w][j][dt * 16 + r16] = o[dt][i];
    }
  }
  __syncthreads();
  // merge the waves in order: each thread owns (head j, column d) pairs
  const size_t rec = HD + 2;
  float* pb = a.part + (((size_t)r * a.Hkv + kvh) * a.nsplit) * grp * rec;
  for (int t = threadIdx.x; t < grp * HD; t += 64 * ATTN_NW) {
    const int j = t / HD, d = t % HD;
    float M = -INFINITY;
#pragma unroll
    for (int q = 0; q < ATTN_NW; ++q) M = fmaxf(M, sM[q][j]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int q = 0; q < ATTN_NW; ++q) {
        const float wgt = sM[q][j] == -INFINITY ? 0.f : __expf(sM[q][j] - M);
        L += wgt * sL[q][j];
        O += wgt * sO[q][j][d];
      }
    }
    if (a.nsplit == 1) {
      Act<T>::put(a.o, r, a.ldo, (kvh * grp + j) * HD + d, L > 0.f ? O / L : 0.f);
    } else {
      float* pj = pb + ((size_t)split * grp + j) * rec;
      pj[d] = O;
      if (d == 0) {
        pj[HD] = M;
        pj[HD + 1] = L;
      }
    }
  }
}

// Log-sum-exp combine of the splits of one (row, head), in split order.
template <typename T>
__global__ __launch_bounds__(64) void k_attn_combine(AttnArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  const int r = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int grp = a.H / a.Hkv, kvh = h / grp, j = h % grp, HD = a.hd;
  const size_t rec = HD + 2;
  const float* pb = a.part + (((size_t)r * a.Hkv + kvh) * a.nsplit) * grp * rec;
  float M = -INFINITY;
  for (int s = 0; s < a.nsplit; ++s) M = fmaxf(M, pb[((size_t)s * grp + j) * rec + HD]);
  for (int d = lane; d < HD; d += 64) {
    float L = 0.f, O = 0.f;
    if (M != -INFINITY) {
      for (int s = 0; s < a.nsplit; ++s) {
        const float* ps = pb + ((size_t)s * grp + j) * rec;
        const float ms = ps[HD];
        const float wgt = ms == -INFINITY ? 0.f : __expf(ms - M);
        L += wgt * ps[HD + 1];
        O += wgt * ps[d];
      }
    }
    Act<T>::put(a.o, r, a.ldo, h * HD + d, L > 0.f ? O / L : 0.f);
  }
}

template <typename T, int HD>
__global__ __launch_bounds__(256) void k_attn_prefill(AttnArgs a) {
  constexpr int EPL = Frag<T>::EPL, KB = Frag<T>::KB, NF = HD / KB, ND = HD / 16;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, r16 = lane & 15, g = lane >> 4;
  const int h = blockIdx.y;
  const int grp = a.H / a.Hkv, kvh = h / grp;
  const int row0 = blockIdx.x * 64 + w * 16;
  if (row0 >= a.R) return;
  const RowInfo r0 = row_info(a.rm, row0);
  const T* Kb = (const T*)a.K + r0.b * a.sb + kvh * a.sh;
  const T* Vb = (const T*)a.VT + r0.b * a.sb + kvh * a.sh;
  const int qrow = row0 + r16;
  const bool qok = qrow < a.R;
  u4 qf[NF], ql[NF];
  constexpr int PL = Act<T>::PL;
  const T* qp = (const T*)a.q + (size_t)(qok ? qrow : row0) * a.ldq * PL + (size_t)h * HD + g * EPL;
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    qf[f] = qok ? ld16(qp + f * KB) : zero16();
    ql[f] = (Act<T>::SPLIT && qok) ? ld16(qp + a.ldq + f * KB) : zero16();
  }
  // causal: row with slot s sees slots [0, s]; rows past the chunk see nothing
  const int limit = qok ? r0.slot + r16 + 1 : 0;
  const int wave_end = r0.slot + min(15, a.R - 1 - row0) + 1;
  f4 o[ND];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) o[dt] = f4{0.f, 0.f, 0.f, 0.f};
  float mrun = -INFINITY, lrun = 0.f;
  const float scale = 1.0f / sqrtf((float)HD);
  // per-lane limit: the score mask uses this lane's query row (r16)
  attn_range<T, HD>(Kb, Vb, a.S, 0, 0, (wave_end + KB - 1) / KB, limit, qf, ql, scale, mrun, lrun, o);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int j = 4 * g + i;  // query row within the wave
    const float lj = __shfl(lrun, j, WAVE);
    if (row0 + j < a.R) {
      const float inv = lj > 0.f ? 1.0f / lj : 0.f;
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) Act<T>::put(a.o, row0 + j, a.ldo, h * HD + r16 + dt * 16, o[dt][i] * inv);
    }
  }
}

template <typename T>
static int decode_t(const AttnArgs& a, Stream s) {
  dim3 grid(a.nsplit, a.Hkv, a.R);
  if (a.hd == 64) hipLaunchKernelGGL((k_attn_decode<T, 64>), grid, dim3(64 * ATTN_NW), 0, s, a);
  else if (a.hd == 128) hipLaunchKernelGGL((k_attn_decode<T, 128>), grid, dim3(64 * ATTN_NW), 0, s, a);
  else return -1;
  if (a.nsplit > 1) hipLaunchKernelGGL((k_attn_combine<T>), dim3(a.R, a.H), dim3(64), 0, s, a);
  return 0;
}
template <typename T>
static int prefill_t(const AttnArgs& a, Stream s) {
  dim3 grid((a.R + 63) / 64, a.H);
  if (a.hd == 64) hipLaunchKernelGGL((k_attn_prefill<T, 64>), grid, dim3(256), 0, s, a);
  else if (a.hd == 128) hipLaunchKernelGGL((k_attn_prefill<T, 128>), grid, dim3(256), 0, s, a);
  else return -1;
  return 0;
}

int launch_attn_decode(int dtype, const AttnArgs& a, Stream s) {
  if (a.H % a.Hkv != 0 || a.H / a.Hkv > 4 || a.S % 64 != 0) return -1;
  return dtype == 1 ? decode_t<bf16>(a, s) : decode_t<float>(a, s);
}
int launch_attn_prefill(int dtype, const AttnArgs& a, Stream s) {
  if (a.H % a.Hkv != 0 || a.S % 64 != 0 || a.rm.mode != ROWS_PREFILL) return -1;
  return dtype == 1 ? prefill_t<bf16>(a, s) : prefill_t<float>(a, s);
}

}  // namespace ham
