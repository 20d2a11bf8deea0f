// Device-side building blocks shared by every kernel of the library (gfx950).
//
// Storage types: `float` (fp32 models) and `bf16` (raw uint16 bit patterns of
// bfloat16).  The matrix-core fragments below are the only place where the two
// differ: one 16-byte load per lane per operand feeds either one
// v_mfma_f32_16x16x32_bf16 (8 bf16 per lane) or four v_mfma_f32_16x16x4_f32
// (4 fp32 per lane).  In both cases lane l of a wave holds operand row (l & 15)
// and the k-slice owned by lane group g = l >> 4; the accumulator holds
// D[4g + i][l & 15], i = 0..3.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ham {

typedef uint16_t bf16;
typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));  // one 16-byte lane fragment

static constexpr int WAVE = 64;

__device__ __forceinline__ float bf2f(bf16 u) { return __uint_as_float(((uint32_t)u) << 16); }

// round to nearest even (values are finite by construction): gfx950's
// v_cvt_pk_bf16_f32, one instruction per pair of values
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ bf16 f2bf(float f) { return __builtin_bit_cast(bf16, (__bf16)f); }
__device__ __forceinline__ uint32_t f2bf2(float lo16, float hi16) {
  return __builtin_bit_cast(uint32_t, bf16x2_t{(__bf16)lo16, (__bf16)hi16});
}

template <typename T> __device__ __forceinline__ float to_f(T v);
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<bf16>(bf16 v) { return bf2f(v); }

template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float v) { return f2bf(v); }

// elements of T in one 16-byte lane fragment, and k covered by one wave fragment
template <typename T> struct Frag;
template <> struct Frag<bf16> {
  static constexpr int EPL = 8;
  static constexpr int KB = 32;
  static __device__ __forceinline__ void mma(f4& acc, const u4& a, const u4& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
  }
};
template <> struct Frag<float> {
  static constexpr int EPL = 4;
  static constexpr int KB = 16;
  static __device__ __forceinline__ void mma(f4& acc, const u4& a, const u4& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
  }
};

// Activation operands of the matrix products (rows of logical width W).
// fp32 models keep fp32 rows.  bf16 models keep each fp32 value v as the bf16
// pair hi = bf16(v), lo = bf16(v - hi) (16 significant bits) in two planes per
// row, [hi 0..W) [lo 0..W), so that each plane loads as 16-byte fragments; a
// product then takes two bf16 matrix-core instructions, hi and lo.
template <typename T> struct Act;
template <> struct Act<float> {
  static constexpr bool SPLIT = false;
  static constexpr int PL = 1;
  static __device__ __forceinline__ void put(void* base, size_t row, int W, int i, float v) {
    ((float*)base)[row * W + i] = v;
  }
};
template <> struct Act<bf16> {
  static constexpr bool SPLIT = true;
  static constexpr int PL = 2;
  static __device__ __forceinline__ void put(void* base, size_t row, int W, int i, float v) {
    bf16* r = (bf16*)base + row * 2 * W;
    const bf16 h = f2bf(v);
    r[i] = h;
    r[W + i] = f2bf(v - bf2f(h));
  }
};

// Fragment-tiled weight layout.  A weight matrix W [N][K] (N a multiple of 16,
// K of the fragment width KB) is stored as 1 KB blocks, one per (16-row tile,
// KB-column fragment), in the order the lanes of a wave read them: lane
// l = 16*g + r holds row r of the tile and elements [g*EPL, g*EPL + EPL) of the
// fragment.  A wave then streams each block with one fully contiguous 1 KB load.
template <typename T>
__host__ __device__ __forceinline__ size_t tiled_index(size_t n, size_t k, size_t K) {
  constexpr int EPL = 16 / sizeof(T), KB = 4 * EPL;
  const size_t nt = n / 16, r = n % 16, f = k / KB, kk = k % KB, g = kk / EPL, e = kk % EPL;
  return ((nt * (K / KB) + f) * 64 + g * 16 + r) * EPL + e;
}

__device__ __forceinline__ u4 ld16(const void* p) { return *reinterpret_cast<const u4*>(p); }
// streamed once per step (weights, KV): non-temporal hint so they do not displace reused lines
__device__ __forceinline__ u4 ld16_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u4*>(p));
}
__device__ __forceinline__ u4 zero16() { return u4{0u, 0u, 0u, 0u}; }

// Raw buffer loads with the hardware range check: a lane whose byte offset lies
// at or past the descriptor's size gets zeros and makes no memory request.  A
// loop of such loads stays free of branches (the compiler can then wait for
// just the loads it needs) without fetching anything for its idle lanes.
// Descriptor word 3 is the gfx9-family default (no format conversion); the
// base must be wave-uniform.
typedef __amdgpu_buffer_rsrc_t BufRsrc;
constexpr uint32_t BUF_OOB = 0xFFFFFFF0u;
__device__ __forceinline__ BufRsrc buf_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ f4 buf_f4(BufRsrc r, uint32_t off) {
  return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ float buf_f1(BufRsrc r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
// streamed (non-temporal) 16-byte load
__device__ __forceinline__ u4 buf_u4_stream(BufRsrc r, uint32_t off) {
  return __builtin_bit_cast(u4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2));
}

// Workgroup barrier for data exchanged through LDS: this wave's LDS accesses
// complete, then s_barrier.  __syncthreads also waits for every vector memory
// operation the wave still has in flight (its release fence must cover global
// stores), prefetched weight blocks included; this one lets them stay in flight.
// Only for exchanges through LDS: global memory written before it is not
// ordered for the other waves.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// pack 8 floats (bf16) / 4 floats (fp32) into one lane fragment
__device__ __forceinline__ u4 pack_frag_bf16(const float* v) {
  return u4{f2bf2(v[0], v[1]), f2bf2(v[2], v[3]), f2bf2(v[4], v[5]), f2bf2(v[6], v[7])};
}

// one product step with an activation fragment pair as the A operand
template <typename T>
__device__ __forceinline__ void mma_act(f4& acc, const u4& xhi, const u4& xlo, const u4& w) {
  Frag<T>::mma(acc, xhi, w);
  if constexpr (Act<T>::SPLIT) Frag<T>::mma(acc, xlo, w);
}
// ... and as the B operand
template <typename T>
__device__ __forceinline__ void mma_act_b(f4& acc, const u4& a, const u4& xhi, const u4& xlo) {
  Frag<T>::mma(acc, a, xhi);
  if constexpr (Act<T>::SPLIT) Frag<T>::mma(acc, a, xlo);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, WAVE));
  return v;
}

// Block-wide sum for blockDim.x == 256 (4 waves); every thread gets the result.
__device__ __forceinline__ float block_sum256(float v, float* sh4) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh4[w] = v;
  __syncthreads();
  return (sh4[0] + sh4[1]) + (sh4[2] + sh4[3]);
}

// any nonzero among n <= 64 flags (one load per lane, then a wave vote; every
// wave of a workgroup reaches the same answer); used to skip work no sequence needs
__device__ __forceinline__ bool any_flag(const int* flags, int n) {
  if (flags == nullptr) return true;
  const int lane = threadIdx.x & 63;
  const int v = lane < n ? flags[lane] : 0;
  return __ballot(v != 0) != 0ull;
}

}  // namespace ham
