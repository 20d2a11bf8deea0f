// Attention over the smashed KV cache (one slot per fused group, Sec. 3.1).
//
// Cache layout per layer: K [seq][kv_head][slot][hd] and V in 32-slot tiles,
// d-major inside a tile ([seq][kv_head][slot/32][hd][32], ham_internal.h), so
// that both products are matrix-core contractions fed by 16-byte contiguous
// loads and the K and V of a 32-slot key block are each one contiguous region:
//   S^T = K Q^T   (A = K rows, B = Q^T)  and  O = P V  (A = P, B = V^T rows).
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
// k_attn_prefill: the q-heads of a kv head over 16-row groups of a prompt chunk,
//   key blocks shared through LDS, causal.
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

// NT: non-temporal loads (decode reads every block once); prefill re-reads each
// block from many waves, so it keeps them cacheable.
template <typename T, int HD, bool NT = true>
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
    for (int f = 0; f < B::NF; ++f) blk.k[t][f] = NT ? ld16_stream(kp + f * KB) : ld16(kp + f * KB);
  }
  // V^T row d = dt*16 + r16 of the block's tile, slots base + g*KB/4 .. (KB <= 32 stays inside one tile)
  const T* vp = Vb + vt_offset(r16, base, HD) + g * (KB / 4);
#pragma unroll
  for (int dt = 0; dt < B::ND; ++dt)
    blk.v[dt] = NT ? ld16_stream(vp + (size_t)dt * 16 * VT_TILE) : ld16(vp + (size_t)dt * 16 * VT_TILE);
}

// Keep the first `keep` elements of a lane fragment, zero the rest.
template <typename T> __device__ __forceinline__ void keep_first(u4& v, int keep);
template <> __device__ __forceinline__ void keep_first<bf16>(u4& v, int keep) {
#pragma unroll
  for (int e = 0; e < 8; ++e)
    if (e >= keep) v[e >> 1] &= (e & 1) ? 0x0000FFFFu : 0xFFFF0000u;
}
template <> __device__ __forceinline__ void keep_first<float>(u4& v, int keep) {
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (e >= keep) v[e] = 0u;
}

// Scores of the 16 operand rows against the block (lane: row r16, slots
// base + g*KB/4 + e), masked at `limit` (the lane's row), then the
// online-softmax update of (m, l, o) and the P.V product.  Values of slots at
// or past `vlimit` (the same for every lane) are zeroed first, so whatever a
// slot past the end holds cannot reach the output.
template <typename T, int HD>
__device__ __forceinline__ void attn_block(KVBlock<T, HD>& blk, int base, int limit, int vlimit, const u4* qf,
                                           const u4* ql, float scale, float& mrun, float& lrun, f4* o) {
  using B = KVBlock<T, HD>;
  constexpr int KB = B::KB, ND = B::ND, TT = B::TT, EPL = Frag<T>::EPL;
  const int lane = threadIdx.x & 63, g = lane >> 4;
  if (base + KB > vlimit) {
    const int keep = min(max(vlimit - (base + g * EPL), 0), EPL);
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) keep_first<T>(blk.v[dt], keep);
  }
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
  // rows whose running maximum did not move have alpha = 1 exactly: the rescale
  // of the output rows is skipped when that holds for every row of the tile
  // (once a row has seen many keys its maximum rarely moves)
  if (__any(mnew != mrun)) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float ai = __shfl(alpha, 4 * g + i, WAVE);
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) o[dt][i] *= ai;
    }
  }
  mrun = mnew;
  u4 phi, plo;
  PFrag<T>::make(p, phi, plo);
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) {
    Frag<T>::mma(o[dt], phi, blk.v[dt]);
    if constexpr (PFrag<T>::TWO) Frag<T>::mma(o[dt], plo, blk.v[dt]);
  }
}

// key blocks a wave keeps in flight at once: 8 KB of K and 8 KB of V (a streaming
// probe and the decode step at 4 x 33K slots both ran about 4% faster with
// 16 KB per wave in flight than with 32 KB)
template <int HD> struct AttnChunk { static constexpr int NB = 128 / HD; };

// Key blocks b0, b0 + BS, b0 + 2 BS, ... below b1, of KB slots from slot0,
// masked at `limit` / `vlimit`.  The blocks go in chunks of NB whose loads are
// all issued before any of them is used, so a chunk costs one memory round trip.
template <typename T, int HD, bool NT = true, int BS = 1>
__device__ __forceinline__ void attn_blocks(const T* Kb, const T* Vb, int S, int slot0, int b0, int b1, int limit,
                                            int vlimit, const u4* qf, const u4* ql, float scale, float& mrun,
                                            float& lrun, f4* o) {
  constexpr int KB = Frag<T>::KB, NB = AttnChunk<HD>::NB;
  for (int c = b0; c < b1; c += NB * BS) {
    KVBlock<T, HD> blk[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i)
      if (c + i * BS < b1) kv_load<T, HD, NT>(blk[i], Kb, Vb, S, slot0 + (c + i * BS) * KB);
#pragma unroll
    for (int i = 0; i < NB; ++i)
      if (c + i * BS < b1)
        attn_block<T, HD>(blk[i], slot0 + (c + i * BS) * KB, limit, vlimit, qf, ql, scale, mrun, lrun, o);
  }
}

constexpr int ATTN_NW = 8;

// Shared state of one (row, kv head, split) workgroup: per wave the softmax
// max, sum and unnormalised output rows of its q-heads, plus an optional extra
// one-slot state (score, value) merged after the waves.
template <int HD>
struct AttnLds {
  float O[ATTN_NW][4][HD];
  float M[ATTN_NW][16], L[ATTN_NW][16];
  float xs[4];      // extra slot: scaled score per q-head
  float xv[HD];     // extra slot: value
};

template <typename T, int HD>
__device__ __forceinline__ void attn_publish(AttnLds<HD>& sh, int grp, float mrun, float lrun, const f4* o) {
  constexpr int ND = HD / 16;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, r16 = lane & 15, g = lane >> 4;
  if (g == 0) {
    sh.M[w][r16] = mrun;
    sh.L[w][r16] = lrun;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int j = 4 * g + i;  // rows 4g+i of the output live in lane group g
    if (j < grp) {
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) sh.O[w][j][dt * 16 + r16] = o[dt][i];
    }
  }
}

// Split records of the decode attention: unnormalised outputs
// [R][Hkv][nsplit][grp][hd], then (max, sum) [R][Hkv][nsplit][grp][2].
__device__ __forceinline__ size_t attn_rec(int r, int kvh, int split, int j, int Hkv, int nsplit, int grp) {
  return (((size_t)r * Hkv + kvh) * nsplit + split) * grp + j;
}

// After a barrier: merge the waves in order (then the extra slot, if any); each
// thread owns (q-head j, column d) pairs.  One split: normalised output; else
// the split's record.
template <typename T, int HD>
__device__ __forceinline__ void attn_merge_store(const AttnLds<HD>& sh, bool extra, int grp, int r, int R, int kvh,
                                                 int split, int nsplit, int Hkv, void* out, int ldo, float* part) {
  for (int t = threadIdx.x; t < grp * HD; t += 64 * ATTN_NW) {
    const int j = t / HD, d = t % HD;
    float M = extra ? sh.xs[j] : -INFINITY;
#pragma unroll
    for (int q = 0; q < ATTN_NW; ++q) M = fmaxf(M, sh.M[q][j]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int q = 0; q < ATTN_NW; ++q) {
        const float wgt = sh.M[q][j] == -INFINITY ? 0.f : __expf(sh.M[q][j] - M);
        L += wgt * sh.L[q][j];
        O += wgt * sh.O[q][j][d];
      }
      if (extra) {
        const float wgt = __expf(sh.xs[j] - M);
        L += wgt;
        O += wgt * sh.xv[d];
      }
    }
    if (nsplit == 1) {
      Act<T>::put(out, r, ldo, (kvh * grp + j) * HD + d, L > 0.f ? O / L : 0.f);
    } else {
      const size_t q = attn_rec(r, kvh, split, j, Hkv, nsplit, grp);
      part[q * HD + d] = O;
      if (d == 0) {
        float* ml = part + (size_t)R * Hkv * nsplit * grp * HD + 2 * q;
        ml[0] = M;
        ml[1] = L;
      }
    }
  }
}

// One workgroup per (query row, kv head, slot split) over a cache that already
// holds every visible slot (the attention op, the micro decoder's first step);
// its waves take consecutive key blocks of the split's slot range.
template <typename T, int HD>
__global__ __launch_bounds__(64 * ATTN_NW) void k_attn_decode(AttnArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  constexpr int EPL = Frag<T>::EPL, KB = Frag<T>::KB, NF = HD / KB, ND = HD / 16;
  __shared__ AttnLds<HD> sh;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, r16 = lane & 15, g = lane >> 4;
  const int split = blockIdx.x, kvh = blockIdx.y, r = blockIdx.z;
  const int grp = a.H / a.Hkv;
  const RowInfo ri = row_info(a.rm, r);
  const int nval = ri.enabled ? ri.n_valid : 0;
  int chunk = (nval + a.nsplit - 1) / a.nsplit;
  chunk = (chunk + KB - 1) / KB * KB;
  const int s0 = split * chunk;
  const int s1 = min(nval, s0 + chunk);
  const int nblk = s1 > s0 ? (s1 - s0 + KB - 1) / KB : 0;
  const int b0 = w * nblk / ATTN_NW, b1 = (w + 1) * nblk / ATTN_NW;
  const T* Kb = (const T*)a.K + ri.b * a.sb + kvh * a.sh;
  const T* Vb = (const T*)a.VT + ri.b * a.sb + kvh * a.sh;
  u4 qf[NF], ql[NF];
  constexpr int PL = Act<T>::PL;
  const T* qp = (const T*)a.q + (size_t)r * (a.q_pitch ? a.q_pitch : a.ldq) * PL + (size_t)(kvh * grp + r16) * HD +
               g * EPL;
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
  attn_blocks<T, HD>(Kb, Vb, a.S, s0, b0, b1, s1, s1, qf, ql, scale, mrun, lrun, o);
  attn_publish<T, HD>(sh, grp, mrun, lrun, o);
  __syncthreads();
  attn_merge_store<T, HD>(sh, false, grp, r, a.R, kvh, split, a.nsplit, a.Hkv, a.o, a.ldo, a.part);
}

// ---------------------------------------------------------------- fused decode step
// One decode row per sequence whose newest slot is produced by this step (the
// base model's fused input, or micro step k >= 2): finishes the q/k/v
// projection (sum of the split-K partials in split order), applies rotate-half
// RoPE to q and k, appends k and v to the cache (split 0 only), and attends
// over the cached slots plus the new one, which enters from registers as an
// extra one-slot softmax state, so no workgroup reads a slot written in the
// same launch.  Key blocks are partitioned statically over the host's bound on
// the cached slots, so their loads need nothing from the per-row state.
//
// RoPE in the fragment layout: lane (r16, g) holds elements f*KB + g*EPL + e of
// fragment f; the rotate-half partner of fragment f < NF/2 is fragment
// f + NF/2 at the same (g, e), so every rotation stays inside one lane.
constexpr int ATTN_STEP_MAXS = 8;  // split-K partials of the projection summed by the step kernel

template <typename T, int HD>
__global__ __launch_bounds__(64 * ATTN_NW) void k_attn_step(AttnStepArgs a) {
  constexpr int EPL = Frag<T>::EPL, KB = Frag<T>::KB, NF = HD / KB, ND = HD / 16, NB = AttnChunk<HD>::NB;
  constexpr int MAXS = ATTN_STEP_MAXS;
  __shared__ AttnLds<HD> sh;
  __shared__ float sraw[6 * HD];  // summed projection: q-heads (grp*HD) | k (HD) | v (HD)
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, r16 = lane & 15, g = lane >> 4;
  const int split = blockIdx.x, kvh = blockIdx.y, r = blockIdx.z;
  const int grp = a.H / a.Hkv;
  const T* Kb = (const T*)a.K + (size_t)r * a.sb + kvh * a.sh;  // decode rows: row r is sequence r
  const T* Vb = (const T*)a.VT + (size_t)r * a.sb + kvh * a.sh;
  // this wave's key blocks.  Split launches: the split's static share of the
  // blocks of [0, kv_cap), so the first loads need nothing from memory.  One
  // workgroup per row: the row's own cached blocks (rows shorter than kv_cap
  // would leave waves idle), at the cost of reading the row's length first.
  int b0, b1;
  RowInfo ri;
  // Wave w takes blocks w, w + NW, w + 2 NW, ... of the range, so at any time
  // the waves of a workgroup read one contiguous window of K and one of V
  // (measured 2.7% faster at 4 x 33K slots than a contiguous sub-range each).
  constexpr int BS = ATTN_NW;
  if (a.nsplit == 1) {
    ri = row_info(a.rm, r);
    b0 = w;
    b1 = (min(max(ri.n_valid - 1, 0), a.kv_cap) + KB - 1) / KB;
  } else {
    const int nblk_all = (a.kv_cap + KB - 1) / KB;
    const int per = (nblk_all + a.nsplit - 1) / a.nsplit;
    const int sb0 = min(nblk_all, split * per);
    b0 = sb0 + w;
    b1 = min(nblk_all, sb0 + per);
  }
  // first chunk of keys in flight before anything else
  KVBlock<T, HD> blk[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i)
    if (b0 + i * BS < b1) kv_load<T, HD>(blk[i], Kb, Vb, a.S, (b0 + i * BS) * KB);
  if (!any_flag(a.gate, a.gate_n)) return;
  if (a.nsplit != 1) ri = row_info(a.rm, r);
  // the projection values of this kv head: one 4-float chunk per thread, all splits
  const int nch = (grp + 2) * HD / 4;
  const int ns = a.part ? a.nsplit_qkv : 1;
  const float* src = a.part ? a.part : a.qkv;
  const size_t sstride = (size_t)a.pM * a.ldqkv;
  if (threadIdx.x < nch) {
    const int c = threadIdx.x * 4;
    int col;
    if (c < grp * HD) col = kvh * grp * HD + c;
    else if (c < (grp + 1) * HD) col = a.H * HD + kvh * HD + (c - grp * HD);
    else col = (a.H + a.Hkv) * HD + kvh * HD + (c - (grp + 1) * HD);
    const float* p = src + (size_t)r * a.ldqkv + col;
    f4 t[MAXS];
#pragma unroll
    for (int s = 0; s < MAXS; ++s)
      if (s < ns) t[s] = *reinterpret_cast<const f4*>(p + (size_t)s * sstride);
    f4 acc = t[0];
#pragma unroll
    for (int s = 1; s < MAXS; ++s)
      if (s < ns) acc += t[s];
#pragma unroll
    for (int e = 0; e < 4; ++e) sraw[c + e] = acc[e];
  }
  // RMSNorm scale of this row when the projection's input was left unscaled
  float rinv = 1.f;
  if (a.ss && a.ss_n <= MAXS) {  // per-split sums of a staged projection
    float sv[MAXS];
#pragma unroll
    for (int s = 0; s < MAXS; ++s) sv[s] = s < a.ss_n ? a.ss[(size_t)s * a.pM + r] : 0.f;
    float ss = 0.f;
#pragma unroll
    for (int s = 0; s < MAXS; ++s) ss += sv[s];
    rinv = 1.0f / sqrtf(ss / (float)a.d + a.eps);
  } else if (a.ss) {  // per column tile sums of a NormOut epilogue (at most 256): each wave sums them
    float sv[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int t = lane + 64 * q;
      sv[q] = t < a.ss_n ? a.ss[(size_t)t * a.pM + r] : 0.f;
    }
    const float ss = wave_sum((sv[0] + sv[1]) + (sv[2] + sv[3]));
    rinv = 1.0f / sqrtf(ss / (float)a.d + a.eps);
  }
  // RoPE factors of this row: elements i = f*KB + g*EPL + e, f < NF/2
  const float* cp = a.cos_p + (size_t)r * a.cs_stride;
  const float* sp = a.sin_p + (size_t)r * a.cs_stride;
  float cs[NF / 2][EPL], sn[NF / 2][EPL];
#pragma unroll
  for (int f = 0; f < NF / 2; ++f)
#pragma unroll
    for (int e4 = 0; e4 < EPL; e4 += 4) {
      const f4 cv = *reinterpret_cast<const f4*>(cp + f * KB + g * EPL + e4);
      const f4 sv = *reinterpret_cast<const f4*>(sp + f * KB + g * EPL + e4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        cs[f][e4 + e] = cv[e];
        sn[f][e4 + e] = sv[e];
      }
    }
  __syncthreads();
  // rotated q (this lane's q-head r16) and k, in fragment order
  float qv[NF][EPL], kv[NF][EPL];
  const int qh = min(r16, grp - 1);
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      qv[f][e] = sraw[qh * HD + f * KB + g * EPL + e] * rinv;
      kv[f][e] = sraw[grp * HD + f * KB + g * EPL + e] * rinv;
    }
#pragma unroll
  for (int f = 0; f < NF / 2; ++f)
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      const float c = cs[f][e], s = sn[f][e];
      const float q1 = qv[f][e], q2 = qv[f + NF / 2][e];
      qv[f][e] = q1 * c - q2 * s;
      qv[f + NF / 2][e] = q2 * c + q1 * s;
      const float k1 = kv[f][e], k2 = kv[f + NF / 2][e];
      // the cache holds k in the storage type: the new slot's score uses that value
      kv[f][e] = to_f<T>(from_f<T>(k1 * c - k2 * s));
      kv[f + NF / 2][e] = to_f<T>(from_f<T>(k2 * c + k1 * s));
    }
  u4 qf[NF], ql[NF];
  float dot = 0.f;
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    if constexpr (Act<T>::SPLIT) {
      float lo[EPL];
      qf[f] = pack_frag_bf16(qv[f]);
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const uint32_t hw = (e & 1) ? (qf[f][e >> 1] >> 16) : (qf[f][e >> 1] & 0xFFFFu);
        lo[e] = qv[f][e] - bf2f((bf16)hw);
      }
      ql[f] = pack_frag_bf16(lo);
    } else {
      qf[f] = u4{__float_as_uint(qv[f][0]), __float_as_uint(qv[f][1]), __float_as_uint(qv[f][2]),
                 __float_as_uint(qv[f][3])};
      ql[f] = qf[f];
    }
    if (r16 >= grp) {  // operand rows past the q-heads of this kv head
      qf[f] = zero16();
      ql[f] = zero16();
    }
#pragma unroll
    for (int e = 0; e < EPL; ++e) dot += qv[f][e] * kv[f][e];
  }
  dot += __shfl_xor(dot, 16, WAVE);
  dot += __shfl_xor(dot, 32, WAVE);
  const float scale = 1.0f / sqrtf((float)HD);
  // the new slot: row checks, cache append (split 0), extra softmax state
  const int cached = ri.n_valid - 1;
  const bool slot_ok = ri.slot == cached && ri.slot >= 0 && ri.slot < a.S && cached <= a.kv_cap;
  const bool extra = split == 0 && ri.enabled && slot_ok;
  if (split == 0 && ri.enabled && !slot_ok && threadIdx.x == 0) atomicOr(a.rm.st.err + r, 8);
  if (extra) {
    if (w == 0 && g == 0 && r16 < grp) sh.xs[r16] = dot * scale;
    if (w == 0 && r16 == 0) {
      T* kd = (T*)a.K + (size_t)r * a.sb + kvh * a.sh + (size_t)ri.slot * HD + g * EPL;
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        u4 pk;
        if constexpr (Act<T>::SPLIT) pk = pack_frag_bf16(kv[f]);
        else pk = u4{__float_as_uint(kv[f][0]), __float_as_uint(kv[f][1]), __float_as_uint(kv[f][2]),
                     __float_as_uint(kv[f][3])};
        *reinterpret_cast<u4*>(kd + f * KB) = pk;
      }
    }
    for (int d = threadIdx.x; d < HD; d += 64 * ATTN_NW) {
      const T v = from_f<T>(sraw[(grp + 1) * HD + d] * rinv);
      sh.xv[d] = to_f<T>(v);
      ((T*)a.VT)[(size_t)r * a.sb + kvh * a.sh + vt_offset(d, ri.slot, HD)] = v;
    }
  }
  // cached slots [0, cached): the first chunk is in registers already
  const int limit = (ri.enabled && slot_ok) ? cached : 0;
  f4 o[ND];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) o[dt] = f4{0.f, 0.f, 0.f, 0.f};
  float mrun = -INFINITY, lrun = 0.f;
#pragma unroll
  for (int i = 0; i < NB; ++i)
    if (b0 + i * BS < b1) attn_block<T, HD>(blk[i], (b0 + i * BS) * KB, limit, limit, qf, ql, scale, mrun, lrun, o);
  // kv_cap bounds every row of the launch; this row's own length ends the loop
  attn_blocks<T, HD, true, BS>(Kb, Vb, a.S, 0, b0 + NB * BS, min(b1, (limit + KB - 1) / KB), limit, limit, qf, ql,
                               scale, mrun, lrun, o);
  attn_publish<T, HD>(sh, grp, mrun, lrun, o);
  __syncthreads();
  attn_merge_store<T, HD>(sh, extra, grp, r, a.R, kvh, split, a.nsplit, a.Hkv, a.o, a.ldo, a.part_out);
}

// Log-sum-exp combine of the splits of one (row, head) (nsplit <= 64): lane s
// of wave 0 holds split s and forms its weight exp(m_s - M) / L with wave
// reductions; then thread t sums the weighted outputs of element t % hd over
// splits t / hd, t / hd + G, ... (G = 256 / hd, all loads of a thread in flight
// together) and the G partial sums are added in order.
constexpr int COMBINE_THREADS = 256;
template <typename T>
__global__ __launch_bounds__(COMBINE_THREADS) void k_attn_combine(AttnArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  __shared__ float wts[64];
  __shared__ float acc[COMBINE_THREADS];
  const int r = blockIdx.x, h = blockIdx.y, tid = threadIdx.x, lane = tid & 63;
  const int grp = a.H / a.Hkv, kvh = h / grp, j = h % grp, HD = a.hd, ns = a.nsplit;
  const float* ml = a.part + (size_t)a.R * a.Hkv * ns * grp * HD;
  if (tid < 64) {
    float ms = -INFINITY, ls = 0.f;
    if (lane < ns) {
      const size_t q = attn_rec(r, kvh, lane, j, a.Hkv, ns, grp);
      ms = ml[2 * q];
      ls = ml[2 * q + 1];
    }
    const float M = wave_max(ms);
    const float e = (ms == -INFINITY) ? 0.f : __expf(ms - M);
    const float L = wave_sum(e * ls);
    if (lane < ns) wts[lane] = L > 0.f ? e / L : 0.f;
  }
  __syncthreads();
  const int G = COMBINE_THREADS / HD, d = tid % HD, sg = tid / HD;
  float o = 0.f;
  if (sg < G) {
    constexpr int UN = 8;
    for (int s0 = sg; s0 < ns; s0 += G * UN) {
      float v[UN];
#pragma unroll
      for (int u = 0; u < UN; ++u) {
        const int sp = s0 + u * G;
        v[u] = sp < ns ? a.part[attn_rec(r, kvh, sp, j, a.Hkv, ns, grp) * HD + d] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < UN; ++u) {
        const int sp = s0 + u * G;
        if (sp < ns) o += wts[sp] * v[u];
      }
    }
  }
  acc[tid] = o;
  __syncthreads();
  if (tid < HD) {
    float x = acc[tid];
    for (int q = 1; q < G; ++q) x += acc[q * HD + tid];
    Act<T>::put(a.o, r, a.ldo, h * HD + tid, x);
  }
}

constexpr int PF_NW = 8, PF_NBL = 2, PF_RT = 2;
#ifndef HAM_PFA_NS
#define HAM_PFA_NS 4
#endif
constexpr int PFA_NS = HAM_PFA_NS;  // stages of key blocks in the LDS ring (PFA_NS - 1 in flight)
template <typename T, int HD>
struct PrefillBlock {  // 1 KB fragments of one key block in LDS: K (tile, fragment), then V (d-tile)
  static constexpr int KB = Frag<T>::KB, EPL = Frag<T>::EPL, NF = HD / KB, ND = HD / 16, TT = KB / 16;
  static constexpr int KF = TT * NF, VF = ND, BF = KF + VF;
  static constexpr int KU = KF * 64, BU = BF * 64;
};

// s_waitcnt with vmcnt <= n (0..63) and lgkmcnt = 0 (expcnt untouched)
template <int N>
__device__ __forceinline__ void pfa_wait_vm_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

// Prefill: causal attention of a prompt chunk (rows of mode PREFILL: slots
// t0 + r of one sequence).  One workgroup of PF_NW waves per (row chunk, kv
// head): wave w takes q-head kvh*grp + w % grp and PF_RT tiles of 16 rows from
// row 16*PF_RT*(w / grp) of the chunk, so a chunk is 16*PF_RT*(PF_NW / grp)
// rows; each key block a wave reads from LDS serves all its row tiles.  Key
// blocks land in LDS straight from memory (global_load_lds_dwordx4), PF_NBL per
// stage in a ring of PFA_NS stages, each 1 KB fragment in the lane order the
// waves read it (K as operand (tile, fragment), V^T as d-tiles), so every
// operand read is one contiguous 1 KB and no registers hold loads in flight.
template <typename T, int HD>
__global__ __launch_bounds__(64 * PF_NW) void k_attn_prefill(AttnArgs a) {
  using PB = PrefillBlock<T, HD>;
  constexpr int KB = PB::KB, EPL = PB::EPL, NF = PB::NF, ND = PB::ND, TT = PB::TT, KU = PB::KU, BU = PB::BU;
  constexpr int BF = PB::BF, SF = PF_NBL * BF;             // fragments per block, per stage
  constexpr int LPW = SF / PF_NW;                          // wave-loads per stage per wave
  static_assert(SF % PF_NW == 0, "stage fragments must split evenly over the waves");
  __shared__ u4 lds[PFA_NS][PF_NBL * BU];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, r16 = lane & 15, g = lane >> 4;
  const int kvh = blockIdx.y;
  const int grp = a.H / a.Hkv, nrg = PF_NW / grp, RB = 16 * PF_RT * nrg;
  const int jh = w % grp, rg = w / grp;
  const int h = kvh * grp + jh;
  const int chunk0 = blockIdx.x * RB;
  if (chunk0 >= a.R) return;  // the same for every wave of the workgroup
  const RowInfo r0 = row_info(a.rm, chunk0);
  const int wg_end = r0.slot + min(RB, a.R - chunk0);  // keys [0, wg_end)
  const int row0 = chunk0 + rg * 16 * PF_RT;
  const bool rows_ok = rg < nrg && row0 < a.R;          // waves past the q-heads only load
  const int wave_end = rows_ok ? r0.slot + (row0 - chunk0) + min(16 * PF_RT, a.R - row0) : 0;
  const T* Kb = (const T*)a.K + r0.b * a.sb + kvh * a.sh;
  const T* Vb = (const T*)a.VT + r0.b * a.sb + kvh * a.sh;

  u4 qf[PF_RT][NF], ql[PF_RT][NF];
  int limit[PF_RT], tile_end[PF_RT];
  constexpr int PL = Act<T>::PL;
#pragma unroll
  for (int t = 0; t < PF_RT; ++t) {
    const int trow = row0 + 16 * t, qrow = trow + r16;
    const bool qok = rows_ok && qrow < a.R;
    const T* qp = (const T*)a.q + (size_t)(qok ? qrow : 0) * a.ldq * PL + (size_t)h * HD + g * EPL;
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      qf[t][f] = qok ? ld16(qp + f * KB) : zero16();
      ql[t][f] = (Act<T>::SPLIT && qok) ? ld16(qp + a.ldq + f * KB) : zero16();
    }
    // causal: the row at slot s sees slots [0, s]
    limit[t] = qok ? r0.slot + (qrow - chunk0) + 1 : 0;
    tile_end[t] = (rows_ok && trow < a.R) ? r0.slot + (trow - chunk0) + min(16, a.R - trow) : 0;
  }

  const int nblk = (wg_end + KB - 1) / KB, nst = (nblk + PF_NBL - 1) / PF_NBL;
  // this wave's fragments of a stage: q = w + PF_NW * i, block q / BF, fragment q % BF.  Lane l of a
  // K fragment (tile t, column fragment f) holds operand row l & 15, whose slot is the one whose score
  // lane group (l & 15) / 4 needs; lane l of a V fragment d-tile dt holds V^T row dt * 16 + (l & 15).
  int koff[LPW], dsto[LPW], blki[LPW];
  bool isk[LPW];
#pragma unroll
  for (int i = 0; i < LPW; ++i) {
    const int q = w + PF_NW * i, j = q % BF;
    blki[i] = q / BF;
    dsto[i] = blki[i] * BU + j * 64;
    isk[i] = j < PB::KF;
    if (isk[i]) {
      const int t = j / NF, f = j % NF, qq = KB / 4;
      const int sl = qq * (r16 / 4) + 4 * t + r16 % 4;
      koff[i] = sl * HD + f * KB + g * EPL;
    } else {
      koff[i] = (j - PB::KF) * 16 + r16;  // V^T row d; its address depends on the block's 32-slot tile
    }
  }
  auto issue = [&](int stg) {  // every wave issues exactly LPW loads per stage (blocks past the end
    u4* slot = lds[stg % PFA_NS];  // re-read the last block, never used), so vmcnt counts stages
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
      const int blk = min(stg * PF_NBL + blki[i], nblk - 1);
      const T* p = isk[i] ? Kb + (size_t)blk * KB * HD + koff[i]
                          : Vb + vt_offset(koff[i], blk * KB, HD) + g * (KB / 4);
      __builtin_amdgcn_global_load_lds((const void*)p, (__attribute__((address_space(3))) void*)(slot + dsto[i]),
                                       16, 0, 0);
    }
  };

  f4 o[PF_RT][ND];
  float mrun[PF_RT], lrun[PF_RT];
#pragma unroll
  for (int t = 0; t < PF_RT; ++t) {
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) o[t][dt] = f4{0.f, 0.f, 0.f, 0.f};
    mrun[t] = -INFINITY;
    lrun[t] = 0.f;
  }
  const float scale = 1.0f / sqrtf((float)HD);
#pragma unroll
  for (int st = 0; st < PFA_NS - 1; ++st)
    if (st < nst) issue(st);
  for (int st = 0; st < nst; ++st) {
    // stage st has landed once at most the loads of the stages issued after it are pending
    if (st + PFA_NS - 2 < nst) pfa_wait_vm_lgkm0<(PFA_NS - 2) * LPW>();
    else pfa_wait_vm_lgkm0<0>();
    asm volatile("s_barrier" ::: "memory");
    // every wave is past stage st - 1: its slot takes stage st + PFA_NS - 1
    if (st + PFA_NS - 1 < nst) issue(st + PFA_NS - 1);
    const u4* sp = lds[st % PFA_NS];
#pragma unroll
    for (int i = 0; i < PF_NBL; ++i) {
      const int blk = st * PF_NBL + i;
      if (blk < nblk && blk * KB < wave_end) {  // blocks past this wave's last row hold nothing it sees
        KVBlock<T, HD> kv;
        const u4* bp = sp + i * BU;
#pragma unroll
        for (int t = 0; t < TT; ++t)
#pragma unroll
          for (int f = 0; f < NF; ++f) kv.k[t][f] = bp[(t * NF + f) * 64 + lane];
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) kv.v[dt] = bp[KU + dt * 64 + lane];
#pragma unroll
        for (int t = 0; t < PF_RT; ++t)
          if (blk * KB < tile_end[t])
            attn_block<T, HD>(kv, blk * KB, limit[t], wave_end, qf[t], ql[t], scale, mrun[t], lrun[t], o[t]);
      }
    }
  }
  if (!rows_ok) return;
#pragma unroll
  for (int t = 0; t < PF_RT; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int jr = 4 * g + i;  // query row within the tile
      const float lj = __shfl(lrun[t], jr, WAVE);
      const int row = row0 + 16 * t + jr;
      if (row < a.R) {
        const float inv = lj > 0.f ? 1.0f / lj : 0.f;
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) Act<T>::put(a.o, row, a.ldo, h * HD + r16 + dt * 16, o[t][dt][i] * inv);
      }
    }
}

template <typename T>
static int decode_t(const AttnArgs& a, Stream s) {
  dim3 grid(a.nsplit, a.Hkv, a.R);
  if (a.hd == 64) launch_k((k_attn_decode<T, 64>), grid, dim3(64 * ATTN_NW), 0, s, a);
  else if (a.hd == 128) launch_k((k_attn_decode<T, 128>), grid, dim3(64 * ATTN_NW), 0, s, a);
  else return -1;
  if (a.nsplit > 1) launch_k((k_attn_combine<T>), dim3(a.R, a.H), dim3(COMBINE_THREADS), 0, s, a);
  return 0;
}
template <typename T>
static int prefill_t(const AttnArgs& a, Stream s) {
  const int grp = a.H / a.Hkv;
  if (grp < 1 || grp > PF_NW) return -1;
  const int rb = 16 * PF_RT * (PF_NW / grp);  // rows per workgroup
  dim3 grid((a.R + rb - 1) / rb, a.Hkv);
  if (a.hd == 64) launch_k((k_attn_prefill<T, 64>), grid, dim3(64 * PF_NW), 0, s, a);
  else if (a.hd == 128) launch_k((k_attn_prefill<T, 128>), grid, dim3(64 * PF_NW), 0, s, a);
  else return -1;
  return 0;
}

template <typename T>
static int step_t(const AttnStepArgs& a, Stream s) {
  dim3 grid(a.nsplit, a.Hkv, a.R);
  if (a.hd == 64) launch_k((k_attn_step<T, 64>), grid, dim3(64 * ATTN_NW), 0, s, a);
  else if (a.hd == 128) launch_k((k_attn_step<T, 128>), grid, dim3(64 * ATTN_NW), 0, s, a);
  else return -1;
  if (a.nsplit > 1 && a.combine) {
    AttnArgs c{};
    c.H = a.H; c.Hkv = a.Hkv; c.hd = a.hd; c.R = a.R; c.nsplit = a.nsplit; c.o = a.o; c.ldo = a.ldo;
    c.part = a.part_out;
    launch_k((k_attn_combine<T>), dim3(a.R, a.H), dim3(COMBINE_THREADS), 0, s, c);
  }
  return 0;
}

int attn_step_max_qkv_split() { return ATTN_STEP_MAXS; }

int launch_attn_step(int dtype, const AttnStepArgs& a, Stream s) {
  if (a.R <= 0) return 0;
  if (a.H % a.Hkv != 0 || a.H / a.Hkv > 4 || a.S % 64 != 0 || a.kv_cap < 0 || a.kv_cap > a.S || a.nsplit < 1 ||
      a.nsplit > 64)  // the split combine holds one split per lane
    return -1;
  if (a.part && (a.nsplit_qkv < 1 || a.nsplit_qkv > ATTN_STEP_MAXS)) return -1;
  if (a.ss && (a.ss_n < 1 || a.ss_n > 256)) return -1;
  if (a.rm.mode != ROWS_DECODE && a.rm.mode != ROWS_MICROK) return -1;
  return dtype == 1 ? step_t<bf16>(a, s) : step_t<float>(a, s);
}

int launch_attn_decode(int dtype, const AttnArgs& a, Stream s) {
  if (a.H % a.Hkv != 0 || a.H / a.Hkv > 4 || a.S % 64 != 0 || a.nsplit < 1 || a.nsplit > 64) return -1;
  return dtype == 1 ? decode_t<bf16>(a, s) : decode_t<float>(a, s);
}
int launch_attn_prefill(int dtype, const AttnArgs& a, Stream s) {
  if (a.H % a.Hkv != 0 || a.S % 64 != 0 || a.rm.mode != ROWS_PREFILL) return -1;
  return dtype == 1 ? prefill_t<bf16>(a, s) : prefill_t<float>(a, s);
}

}  // namespace ham
