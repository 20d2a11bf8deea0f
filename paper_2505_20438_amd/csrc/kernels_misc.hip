// Elementwise and bookkeeping kernels of the decode loop: RMSNorm, RoPE with
// the KV append, the compositional embedder's small pieces, the macro-step and
// prefill set-up of per-sequence state, the micro-decoder input rows, and the
// seeded weight initialiser.
#include <math.h>

#include "device_common.h"
#include "ham_internal.h"
#include "kernels_misc.h"
#include "rows.h"

namespace ham {

// ---------------------------------------------------------------- RMSNorm
// out[r] = g * x / sqrt(mean(x^2) + eps), rounded to the storage type (the GEMM operand)
// A pending split-K result of the previous GEMM (partials) is first added to the
// residual row in split order, and the updated row optionally copied out.  One
// 1024-thread block per row: every thread owns d/1024 columns and issues all of
// its partial loads before summing them.
constexpr int NORM_THREADS = 1024;
constexpr int NORM_MAXV = 8;   // d <= 8192
constexpr int NORM_MAXS = 16;  // pending split-K partials

template <typename T>
__global__ __launch_bounds__(NORM_THREADS) void k_rmsnorm(NormArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  __shared__ float sh[NORM_THREADS / 64];
  const int r = blockIdx.x;
  const int xr = r * a.row_stride + a.row_off;
  float* x = a.x + (size_t)xr * a.ldx;
  float v[NORM_MAXV];
  float ss = 0.f;
#pragma unroll
  for (int e = 0; e < NORM_MAXV; ++e) {
    const int i = threadIdx.x + e * NORM_THREADS;
    v[e] = 0.f;
    if (i < a.d) v[e] = x[i];
  }
  if (a.part) {
    // per element, all partial loads in flight before they are added in split order
    const size_t sstride = (size_t)a.pM * a.ldx;
    const float* pp = a.part + (size_t)xr * a.ldx;
    const int ns = a.nsplit;
#pragma unroll
    for (int e = 0; e < NORM_MAXV; ++e) {
      const int i = threadIdx.x + e * NORM_THREADS;
      if (i < a.d) {
        float p[NORM_MAXS];
#pragma unroll
        for (int q = 0; q < NORM_MAXS; ++q)
          if (q < ns) p[q] = pp[(size_t)q * sstride + i];
#pragma unroll
        for (int q = 0; q < NORM_MAXS; ++q)
          if (q < ns) v[e] += p[q];
        x[i] = v[e];
      }
    }
  }
#pragma unroll
  for (int e = 0; e < NORM_MAXV; ++e) {
    const int i = threadIdx.x + e * NORM_THREADS;
    if (i < a.d) {
      if (a.ctx) a.ctx[(size_t)r * a.ldctx + i] = v[e];
      ss += v[e] * v[e];
    }
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int q = 0; q < NORM_THREADS / 64; ++q) tot += sh[q];
  const float inv = 1.0f / sqrtf(tot / (float)a.d + a.eps);
#pragma unroll
  for (int e = 0; e < NORM_MAXV; ++e) {
    const int i = threadIdx.x + e * NORM_THREADS;
    if (i < a.d) {
      const float o = v[e] * inv * a.g[i];
      Act<T>::put(a.out, r, a.ldo, i, o);
      if (a.hid) a.hid[(size_t)r * a.ldh + i] = o;
    }
  }
}

// Two-phase form for batches of rows (one workgroup per row leaves most CUs
// idle while it reads the pending partials): phase 1 over (256-column chunks,
// rows) folds the partials into x and writes each chunk's sum of squares;
// phase 2 sums a row's chunk sums in order and writes the scaled operand.
constexpr int NORM2_MIN_ROWS = 16, NORM2_MAX_ROWS = 256;  // decode batches (prefill chunks fill the GPU already)
__global__ __launch_bounds__(256) void k_norm_reduce(NormArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  __shared__ float sh4[4];
  const int r = blockIdx.y, i = blockIdx.x * 256 + threadIdx.x;
  const int xr = r * a.row_stride + a.row_off;
  float* x = a.x + (size_t)xr * a.ldx;
  float v = 0.f;
  if (i < a.d) {
    v = x[i];
    if (a.part) {
      const size_t sstride = (size_t)a.pM * a.ldx;
      const float* pp = a.part + (size_t)xr * a.ldx + i;
      float p[NORM_MAXS];
#pragma unroll
      for (int q = 0; q < NORM_MAXS; ++q)
        if (q < a.nsplit) p[q] = pp[(size_t)q * sstride];
#pragma unroll
      for (int q = 0; q < NORM_MAXS; ++q)
        if (q < a.nsplit) v += p[q];
      x[i] = v;
    }
    if (a.ctx) a.ctx[(size_t)r * a.ldctx + i] = v;
  }
  const float ss = block_sum256(v * v, sh4);
  if (threadIdx.x == 0) a.ss[(size_t)r * gridDim.x + blockIdx.x] = ss;
}

template <typename T>
__global__ __launch_bounds__(256) void k_norm_scale(NormArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  const int r = blockIdx.y, i = blockIdx.x * 256 + threadIdx.x, nch = gridDim.x;
  const int xr = r * a.row_stride + a.row_off;
  const float v = i < a.d ? a.x[(size_t)xr * a.ldx + i] : 0.f;
  float tot = 0.f;
  for (int c = 0; c < nch; ++c) tot += a.ss[(size_t)r * nch + c];
  const float inv = 1.0f / sqrtf(tot / (float)a.d + a.eps);
  if (i < a.d) {
    const float o = v * inv * a.g[i];
    Act<T>::put(a.out, r, a.ldo, i, o);
    if (a.hid) a.hid[(size_t)r * a.ldh + i] = o;
  }
}

int launch_norm_reduce(const NormArgs& a, Stream s) {
  // first phase only (x += partials, ctx copy, chunk sums of squares): the
  // batched GEMM that consumes the rows applies 1/rms and the gain itself
  if (a.R < NORM2_MIN_ROWS || a.R > NORM2_MAX_ROWS || !a.ss || a.row_stride != 1 || a.row_off != 0 || a.hid)
    return -1;
  if (a.part && (a.nsplit < 1 || a.nsplit > NORM_MAXS)) return -1;
  launch_k(k_norm_reduce, dim3((a.d + 255) / 256, a.R), dim3(256), 0, s, a);
  return 0;
}

int launch_rmsnorm(int dtype, const NormArgs& a, Stream s) {
  if (a.R <= 0) return 0;
  if (a.d > NORM_THREADS * NORM_MAXV || (a.part && (a.nsplit < 1 || a.nsplit > NORM_MAXS))) return -1;
  if (a.ss && a.R >= NORM2_MIN_ROWS && a.R <= NORM2_MAX_ROWS) {
    const dim3 grid((a.d + 255) / 256, a.R);
    launch_k(k_norm_reduce, grid, dim3(256), 0, s, a);
    if (dtype == 1) launch_k((k_norm_scale<bf16>), grid, dim3(256), 0, s, a);
    else launch_k((k_norm_scale<float>), grid, dim3(256), 0, s, a);
    return 0;
  }
  if (dtype == 1) launch_k((k_rmsnorm<bf16>), dim3(a.R), dim3(NORM_THREADS), 0, s, a);
  else launch_k((k_rmsnorm<float>), dim3(a.R), dim3(NORM_THREADS), 0, s, a);
  return 0;
}

// ---------------------------------------------------------------- RoPE + KV append
// Rotate-half RoPE of q and k at the row's position; q -> q buffer, k -> K cache
// slot, v -> its column of the slot's V tile.  One block per (head of q|k|v, row).
template <typename T>
__global__ __launch_bounds__(64) void k_rope_append(RopeArgs a) {
  if (!any_flag(a.gate, a.gate_n)) return;
  const int hh = blockIdx.x, r = blockIdx.y;
  const int half = a.hd / 2;
  const RowInfo ri = row_info(a.rm, r);
  const float* src = a.qkv + (size_t)r * a.ldqkv + (size_t)hh * a.hd;
  const bool okpos = ri.pos >= 0 && ri.pos < a.max_pos;
  const bool okslot = ri.slot >= 0 && ri.slot < a.S;
  if (!(okpos && okslot)) {
    if (threadIdx.x == 0 && ri.enabled) atomicOr(a.rm.st.err + ri.b, 1);
    return;
  }
  for (int i = threadIdx.x; i < half; i += 64) {
    float x1, x2;
    if (a.part) {  // sum the split-K partials of the projection in split order
      x1 = x2 = 0.f;
      const size_t col = (size_t)hh * a.hd + i;
      for (int s = 0; s < a.nsplit; ++s) {
        const float* ps = a.part + ((size_t)s * a.R + r) * a.ldqkv + col;
        x1 += ps[0];
        x2 += ps[half];
      }
    } else {
      x1 = src[i];
      x2 = src[i + half];
    }
    if (hh < a.H + a.Hkv) {
      const float c = a.cos_t[(size_t)ri.pos * half + i], sn = a.sin_t[(size_t)ri.pos * half + i];
      const float y1 = x1 * c - x2 * sn, y2 = x2 * c + x1 * sn;
      if (hh < a.H) {
        Act<T>::put(a.q, r, a.ldq, hh * a.hd + i, y1);
        Act<T>::put(a.q, r, a.ldq, hh * a.hd + i + half, y2);
      } else if (ri.enabled) {
        T* k = (T*)a.K + ri.b * a.sb + (hh - a.H) * a.sh + (size_t)ri.slot * a.hd;
        k[i] = from_f<T>(y1);
        k[i + half] = from_f<T>(y2);
      }
    } else if (ri.enabled) {
      T* v = (T*)a.VT + ri.b * a.sb + (hh - a.H - a.Hkv) * a.sh;
      v[vt_offset(i, ri.slot, a.hd)] = from_f<T>(x1);
      v[vt_offset(i + half, ri.slot, a.hd)] = from_f<T>(x2);
    }
  }
}

int launch_rope_append(int dtype, const RopeArgs& a, Stream s) {
  if (a.R <= 0) return 0;
  dim3 grid(a.H + 2 * a.Hkv, a.R);
  if (dtype == 1) launch_k((k_rope_append<bf16>), grid, dim3(64), 0, s, a);
  else launch_k((k_rope_append<float>), grid, dim3(64), 0, s, a);
  return 0;
}

// ---------------------------------------------------------------- macro-step set-up
// For each sequence: consume the previous group (fuse it or bypass), advance the
// position by the group size (the fused input sits at its last token's position,
// Sec. 3.2), take the next KV slot, and open a new group.
template <typename T>
__global__ __launch_bounds__(256) void k_macro_begin(MacroArgs a) {
  __shared__ int sh[7];  // n, on, new position, tokens 0..3
  const int b = blockIdx.x, tid = threadIdx.x;
  const SeqPtrs& st = a.st;
  if (tid == 0) {  // every state word in one round trip (tokens past the group are not used)
    const int done = st.done[b], n = st.grp_n[b], pl = st.pos_last[b];
    int t[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) t[j] = st.grp_tok[b * 4 + j];
    sh[0] = n;
    sh[1] = done ? 0 : 1;
    sh[2] = pl + n;  // the fused input sits at its group's last token's position
#pragma unroll
    for (int j = 0; j < 4; ++j) sh[3 + j] = j < n ? t[j] : 0;
  }
  __syncthreads();
  const int n = sh[0], on = sh[1], p = sh[2];
  const int spos = on ? min(max(p, 0), a.max_pos - 1) : -1;
  const int d = a.d, half = a.hd / 2;
  const T* E = (const T*)a.E;
  const T* P = (const T*)a.P;
  // RoPE factors of this step's base input (read by every layer's attention step),
  // loaded together with the embedding rows
  if (spos >= 0)
    for (int i = tid; i < half; i += 256) {
      a.rope_cs[(size_t)b * a.hd + i] = a.cos_t[(size_t)spos * half + i];
      a.rope_cs[(size_t)b * a.hd + half + i] = a.sin_t[(size_t)spos * half + i];
    }
  if (on && n == 1) {  // bypass: the single token's embedding is the base input
    constexpr int U = 8;
    const T* er = E + (size_t)sh[3] * d;
    for (int i0 = tid; i0 < d; i0 += 256 * U) {
      float v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = i0 + 256 * u < d ? to_f<T>(er[i0 + 256 * u]) : 0.f;
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (i0 + 256 * u < d) a.x[(size_t)b * a.ldx + i0 + 256 * u] = v[u];
    }
  } else if (on && n > 1) {
    // e_j = E[t_j] + P[j]; query = mean_j e_j; rows of the embedder's projection GEMM
    constexpr int U = 2;
    for (int i0 = tid; i0 < d; i0 += 256 * U) {
      float ev[U][4], pv[U][4];
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int i = i0 + 256 * u;
          const bool ok = i < d && j < n;
          ev[u][j] = ok ? to_f<T>(E[(size_t)sh[3 + j] * d + i]) : 0.f;
          pv[u][j] = ok ? to_f<T>(P[(size_t)j * d + i]) : 0.f;
        }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + 256 * u;
        if (i >= d) continue;
        float sum = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float e = j < n ? ev[u][j] + pv[u][j] : 0.f;
          sum += e;
          Act<T>::put(a.emb_in, (size_t)b * 5 + 1 + j, d, i, e);
        }
        Act<T>::put(a.emb_in, (size_t)b * 5, d, i, sum / (float)n);
      }
    }
  }
  if (tid == 0) {
    st.step_on[b] = on;
    st.fused[b] = (on && n > 1) ? n : 0;
    if (on) {
      st.pos_last[b] = p;
      st.cur_pos[b] = p;
      st.cur_slot[b] = st.kv_len[b];
      st.kv_len[b] += 1;
      if (p < 0 || p >= a.max_pos) atomicOr(st.err + b, 1);
    }
    st.forced[b] = a.forced_in ? a.forced_in[b] : a.G;
    for (int j = 0; j < 4; ++j) {
      st.teacher[b * 4 + j] = a.teacher_in ? a.teacher_in[b * 4 + j] : 0;
      a.out_tokens[b * 4 + j] = -1;
    }
    a.out_lens[b] = 0;
    st.grp_n[b] = 0;
    st.active[b] = on;
  }
}

// Embedder attention over the <= 4 token rows of a fused group: per head, the
// mean query attends to the rows' keys (Sec. 3.2).  proj = [B*5][3d] fp32 rows
// (row 0 query, rows 1..4 tokens; columns Q | K | V).
template <typename T>
__global__ __launch_bounds__(64) void k_embed_attn(EmbedAttnArgs a) {
  const int b = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int n = a.fused[b];
  if (n < 2) return;
  const int hd = a.hd, HD = a.H * a.hd;  // proj row: Q | K | V blocks of H*hd each
  // lane holds elements lane and lane + 64 of the head: the query, the n keys and
  // values, each summed over the split-K partials (one load of every value per split)
  constexpr int NE = 2;  // hd <= 128
  const int ns = a.part ? a.nsplit : 1;
  const float* src = a.part ? a.part : a.proj;
  const size_t sstride = (size_t)a.B * 5 * 3 * HD;
  float q[NE] = {}, k[4][NE] = {}, v[4][NE] = {};
  for (int sp = 0; sp < ns; ++sp) {
    const float* base = src + (size_t)sp * sstride + (size_t)b * 5 * 3 * HD + (size_t)h * hd;
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      const int i = lane + 64 * e;
      if (i >= hd) continue;
      q[e] += base[i];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (j < n) {
          k[j][e] += base[(size_t)(1 + j) * 3 * HD + HD + i];
          v[j][e] += base[(size_t)(1 + j) * 3 * HD + 2 * HD + i];
        }
    }
  }
  float w[4];
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < NE; ++e) s += q[e] * k[j][e];
    s = wave_sum(s) * (1.0f / sqrtf((float)hd));
    w[j] = j < n ? s : -INFINITY;
    m = fmaxf(m, w[j]);
  }
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    w[j] = j < n ? expf(w[j] - m) : 0.f;
    sum += w[j];
  }
#pragma unroll
  for (int e = 0; e < NE; ++e) {
    const int i = lane + 64 * e;
    if (i >= hd) continue;
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (j < n) acc += w[j] * v[j][e];
    Act<T>::put(a.out, b, HD, h * hd + i, acc / sum);
  }
}

// ---------------------------------------------------------------- prefill set-up
__global__ void k_prefill_begin(PrefillArgs a) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= a.B) return;
  const SeqPtrs& st = a.st;
  const int plast = a.pos_in ? a.pos_in[(size_t)b * a.ldpos + a.P - 1] : a.P - 1;
  st.kv_len[b] = a.P;
  st.pos_last[b] = plast;
  st.cur_pos[b] = plast;
  st.cur_slot[b] = a.P - 1;
  st.emitted[b] = 0;
  st.done[b] = 0;
  st.groups[b] = 0;
  for (int j = 0; j < 5; ++j) st.hist[b * 5 + j] = 0;
  st.step_on[b] = 1;
  st.fused[b] = 0;
  st.grp_n[b] = 0;
  st.active[b] = 1;
  st.err[b] = 0;
  st.forced[b] = a.forced_in ? a.forced_in[b] : a.G;
  for (int j = 0; j < 4; ++j) {
    st.teacher[b * 4 + j] = a.teacher_in ? a.teacher_in[b * 4 + j] : 0;
    a.out_tokens[b * 4 + j] = -1;
  }
  a.out_lens[b] = 0;
}

template <typename T>
__global__ __launch_bounds__(256) void k_gather_rows(GatherArgs a) {
  const int r = blockIdx.x;
  if (a.rows) {
    for (int i = threadIdx.x; i < a.d; i += 256) a.x[(size_t)r * a.ldx + i] = a.rows[(size_t)r * a.d + i];
    return;
  }
  int t = a.ids[r];
  if (t < 0 || t >= a.V) {  // caller-provided id out of range: flag it, read row 0
    if (threadIdx.x == 0) atomicOr(a.err, 2);
    t = 0;
  }
  const T* E = (const T*)a.E;
  for (int i = threadIdx.x; i < a.d; i += 256) a.x[(size_t)r * a.ldx + i] = to_f<T>(E[(size_t)t * a.d + i]);
}

__global__ __launch_bounds__(256) void k_copy_row(const float* src, float* dst, int d) {
  for (int i = threadIdx.x; i < d; i += 256) dst[i] = src[i];
}

// dst row r = src row r (rows of d floats, d % 4 == 0, at their own pitches)
__global__ __launch_bounds__(256) void k_copy_rows(const float* src, long long ld_src, float* dst, long long ld_dst,
                                                   int d) {
  const float* s = src + (size_t)blockIdx.x * ld_src;
  float* t = dst + (size_t)blockIdx.x * ld_dst;
  for (int i = 4 * threadIdx.x; i < d; i += 4 * 256) *reinterpret_cast<f4*>(t + i) = *reinterpret_cast<const f4*>(s + i);
}

// ---------------------------------------------------------------- weight generator
// SplitMix64 (Steele, Lea, Flood 2014): i-th output of the stream seeded with s.
__device__ __forceinline__ uint64_t sm64(uint64_t s, uint64_t i) {
  uint64_t z = s + (i + 1ull) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Box-Muller (cosine branch) in float64, scaled by 0.02, rounded to fp32 then T.
template <typename T>
__global__ __launch_bounds__(256) void k_gen_normal(GenArgs a) {
  const long long count = (long long)a.rows * a.cols;
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < count; i += (long long)gridDim.x * 256) {
    const uint64_t r1 = sm64(a.key, 2ull * (uint64_t)i), r2 = sm64(a.key, 2ull * (uint64_t)i + 1ull);
    const double u1 = ((double)(r1 >> 11) + 1.0) * 0x1p-53;
    const double u2 = (double)(r2 >> 11) * 0x1p-53;
    const double rad = sqrt(-2.0 * log(u1));
    const double ang = (2.0 * 3.141592653589793) * u2;
    const double nv = rad * cos(ang);
    const float v = (float)(nv * 0.02);
    const long long row = i / a.cols, col = i % a.cols;
    long long drow = row + a.row_off;
    // gate and up rows interleaved in blocks of 8: one 16-row tile holds gate and up of 8 features
    if (a.interleave) drow = 16 * (row / 8) + (row % 8) + (a.interleave == 2 ? 8 : 0) + a.row_off;
    const size_t dst = a.tiled ? tiled_index<T>((size_t)drow, (size_t)col, (size_t)a.cols)
                               : (size_t)drow * a.cols + col;
    ((T*)a.dst)[dst] = from_f<T>(v);
  }
}

__global__ void k_fill_f32(float* p, long long n, float v) {
  for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long long)gridDim.x * 256) p[i] = v;
}

// ---------------------------------------------------------------- launchers
#define HAM_T_LAUNCH(dtype, kern, grid, block, s, arg)                           \
  do {                                                                           \
    if ((dtype) == 1) launch_k((kern<bf16>), grid, block, 0, s, arg);  \
    else launch_k((kern<float>), grid, block, 0, s, arg);              \
  } while (0)

void launch_macro_begin(int dtype, const MacroArgs& a, Stream s) {
  HAM_T_LAUNCH(dtype, k_macro_begin, dim3(a.B), dim3(256), s, a);
}
void launch_embed_attn(int dtype, const EmbedAttnArgs& a, Stream s) {
  HAM_T_LAUNCH(dtype, k_embed_attn, dim3(a.B, a.H), dim3(64), s, a);
}
void launch_prefill_begin(const PrefillArgs& a, Stream s) {
  launch_k(k_prefill_begin, dim3((a.B + 255) / 256), dim3(256), 0, s, a);
}
void launch_gather_rows(int dtype, const GatherArgs& a, Stream s) {
  HAM_T_LAUNCH(dtype, k_gather_rows, dim3(a.R), dim3(256), s, a);
}
void launch_copy_row(const float* src, float* dst, int d, Stream s) {
  launch_k(k_copy_row, dim3(1), dim3(256), 0, s, src, dst, d);
}
int launch_copy_rows(const float* src, long long ld_src, float* dst, long long ld_dst, int R, int d, Stream s) {
  if (R < 0 || d % 4 != 0 || ld_src % 4 != 0 || ld_dst % 4 != 0) return -1;
  if (R > 0) launch_k(k_copy_rows, dim3(R), dim3(256), 0, s, src, ld_src, dst, ld_dst, d);
  return 0;
}
void launch_gen_normal(int dtype, const GenArgs& a, Stream s) {
  const long long count = (long long)a.rows * a.cols;
  long long blocks = (count + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  HAM_T_LAUNCH(dtype, k_gen_normal, dim3((unsigned)blocks), dim3(256), s, a);
}
void launch_fill_f32(float* p, long long n, float v, Stream s) {
  long long blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  launch_k(k_fill_f32, dim3((unsigned)blocks), dim3(256), 0, s, p, n, v);
}

}  // namespace ham
