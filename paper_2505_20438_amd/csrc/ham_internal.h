// Internal interfaces between the host orchestration (ham.cpp) and the kernels.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ham {

// Optional timing of the next kernel launch.  When armed, the launch helper
// attaches the two events to the kernel's dispatch itself (its start and end,
// without the queueing before it), then disarms.  One per host thread.
struct LaunchTiming {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchTiming& launch_timing();

template <typename... KArgs, typename... Args>
inline void launch_k(void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t lds, hipStream_t s, Args... args) {
  LaunchTiming& t = launch_timing();
  if (t.start) {
    hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)lds, s, t.start, t.stop, 0u, args...);
    t = LaunchTiming{};
  } else {
    hipLaunchKernelGGL(kernel, grid, block, lds, s, args...);
  }
}

// ---------------------------------------------------------------- KV cache layout
// K [seq][kv_head][slot][hd] (slot-major).  V in tiles of VT_TILE slots, d-major
// inside a tile: [seq][kv_head][slot / VT_TILE][hd][VT_TILE], so the values of
// one 32-slot key block are one contiguous region, like its keys.
constexpr int VT_TILE = 32;
__host__ __device__ __forceinline__ size_t vt_offset(int d, int slot, int hd) {
  return ((size_t)(slot / VT_TILE) * hd + d) * VT_TILE + slot % VT_TILE;
}

// ---------------------------------------------------------------- per-sequence state
// Structure-of-arrays in the state buffer, each int32 [max_batch] (grp_tok, teacher:
// [max_batch][4], hist: [max_batch][5]).
struct SeqPtrs {
  int* kv_len;     // base KV slots held
  int* pos_last;   // RoPE position of the newest base input
  int* cur_pos;    // position of this step's base input
  int* cur_slot;   // KV slot written by this step
  int* emitted;    // tokens emitted so far
  int* budget;     // token budget (0 = none)
  int* done;       // budget spent
  int* groups;     // groups emitted
  int* hist;       // [B][5] group-length histogram
  int* step_on;    // sequence runs this macro-step
  int* fused;      // this step's input is a fused group (n > 1)
  int* active;     // still waiting for the next micro decision
  int* grp_n;      // tokens in the current group
  int* grp_tok;    // [B][4] current group
  int* forced;     // forced length for this step (FORCED mode)
  int* teacher;    // [B][4] teacher tokens for this step
  int* err;        // device-side bounds-check flags
};

// how the rows of a launch map onto sequences, KV slots and positions
enum RowMode { ROWS_PREFILL = 0, ROWS_DECODE = 1, ROWS_MICRO1 = 2, ROWS_MICROK = 3 };
struct RowMap {
  int mode;
  int b;        // PREFILL: the sequence
  int t0;       // PREFILL: slot of row 0
  const int* pos; int ldpos;  // PREFILL: RoPE position of slot t at pos[b*ldpos + t] (null: position = slot)
  int C;        // MICRO*: context rows
  int k;        // MICROK: micro step index (>= 2)
  SeqPtrs st;
};

// ---------------------------------------------------------------- GEMM
enum EpiKind { EPI_F32 = 0, EPI_OP = 1, EPI_RESID = 2, EPI_SWIGLU = 3, EPI_ARGMAX = 4, EPI_XMASK = 5 };

struct DecideArgs {
  SeqPtrs st;
  int B, k, mode, stop_id, G, V, has_teacher;
  float tau;
  int* out_tokens;   // [B][4]
  int* out_lens;     // [B]
  float* dbg_logits; // [B][V] for this k, or null
  float* dbg_stop;   // [B] for this k, or null
  float* stop_buf;   // [B] stop logits (workspace)
  float* best_val;   // [B][ntiles] argmax partials per column tile (a row's are contiguous)
  int* best_idx;
  int ntiles;
  // inputs of micro step prep_k (0: none) for the sequences still running:
  // step 1 = [ctx_1..ctx_C, E[t_0]] per sequence, step k = E[t_{k-1}]
  int prep_k, C, d;
  const float* ctx;  // [B][C][d]
  const void* E;     // embedding table
  float* x;          // [rows][d]
};

// Where the skinny GEMM takes its X operand from.  XS_ACT: activation rows in
// memory (storage-type planes).  The other two build X in LDS in a prologue of
// the GEMM itself (rows M <= 8), so the kernel that would otherwise produce X
// disappears from the launch sequence:
//  XS_NORM: X = g * (x + pending split-K partials) * rinv, the RMSNorm of the
//    updated residual.  With one k-split the workgroup sees the whole row and
//    applies rinv itself; with several, X is left unscaled, each split reports
//    the sum of squares of its k-range in ss_out, and the consumer of the
//    output applies rinv.  Column tile 0 writes the updated rows to x_out
//    (never x itself: other workgroups are still reading it) and to ctx.
//  XS_ATTN: X = attention output combined from the split records of the
//    decode attention (log-sum-exp weights per head, splits in order).
//  XS_NORMW (batched GEMM, 8 < M <= 256): X = g * x * rinv from fp32 rows x whose
//    pending partials the norm's first phase has already folded in; rinv from
//    that phase's 256-column chunk sums of squares ssw [M][nchw].
enum XSource { XS_ACT = 0, XS_NORM = 1, XS_ATTN = 2, XS_NORMW = 3 };
struct XStage {
  const float* x; int ldx;             // NORM: residual rows [M][ldx]
  const float* part; int nsplit, pM;   // NORM: pending partials [nsplit][pM][ldx], or null
  const float* g; float eps;           // NORM: gain [K]
  float* x_out;                        // NORM: updated rows [M][ldx]
  float* ctx; int ldctx;               // NORM: optional copy of the updated rows
  float* ss_out;                       // NORM, k-split launches: [split][M] sums of squares
  const float* rec_o;                  // ATTN: unnormalised outputs [M][Hkv][ans][grp][hd]
  const float* rec_ml;                 // ATTN: (max, sum) [M][Hkv][ans][grp][2]
  int ans, Hkv, grp, hd;               // ATTN: splits, heads, head dim
  const float* ssw; int nchw;          // NORMW: chunk sums of squares [M][nchw]
};

// RESID, unsplit (gemm_norm_out_fits): the next RMSNorm's first half in the
// epilogue.  With x the updated residual rows, writes g * x as the next GEMM's
// operand and, per column tile t, the sums of squares of its columns per row;
// the consumer applies 1/rms (RowScale, or the fused attention step).
struct NormOut {
  const float* g;                  // next norm's gain [N], or null (operand not written)
  void* act; int lda;              // g * x, operand layout [M][lda] (storage type)
  float* ss;                       // [tile][M] sums of squares; null: plain RESID
};

// SWIGLU: the product's rows scaled by 1/rms before the activation, from the
// per-tile sums of squares a NormOut epilogue wrote (n tiles, n <= 256).
struct RowScale {
  const float* ss; int n, d;       // ss [n][M]; rinv = 1/sqrt(sum / d + eps); null: no scaling
  float eps;
};

struct GemmArgs {
  const void* W; int N, K;         // W [N][K] row-major (storage type), N % 32 == 0
  const void* X; int ldx; int M;   // X [M][ldx] (storage type)
  void* out; int ldo;              // destination (see EpiKind)
  float* ctx; int ldctx;           // RESID with NormOut: copy of updated rows (optional)
  const int* rowmask;              // XMASK: rows to store
  const int* gate; int gate_n;     // launch does nothing unless a gate flag is set
  float* part; int* counters; int nsplit;  // split-K partials [nsplit][M][N] (written when nsplit > 1)
  DecideArgs dec;                  // ARGMAX only
  int xsrc; XStage xs;             // X operand source (XS_ACT: X above)
  NormOut no;                      // RESID only
  RowScale rs;                     // SWIGLU only
};

// ---------------------------------------------------------------- attention
struct AttnArgs {
  const void* q; int ldq;          // q [R][H*hd] (storage type), RoPE applied
  int q_pitch;                     // decode: row r of q at r * q_pitch values (0: ldq, rows packed)
  const void* K; const void* VT;   // K [b][Hkv][S][hd], V tiled [b][Hkv][S/32][hd][32] (vt_offset)
  long long sb, sh;                // element strides per sequence and per kv head (both caches)
  int S;                           // slot capacity (row length of VT)
  int H, Hkv, hd, R, nsplit;
  void* o; int ldo;                // o [R][H*hd] (storage type)
  float* part; int* counters;      // split records: outputs [R][Hkv][nsplit][grp][hd], then (max, sum) [..][2]
  RowMap rm;
  const int* gate; int gate_n;
};

// Fused decode step (rows of mode DECODE or MICROK): projection finish, RoPE,
// KV append of the new slot and attention over the cache plus that slot.
struct AttnStepArgs {
  const float* qkv; const float* part; int nsplit_qkv, pM, ldqkv;  // projection [R][ldqkv] or partials [ns][pM][ldqkv]
  const float* cos_p; const float* sin_p; long long cs_stride;     // RoPE factors of row r at +r*cs_stride (hd/2 each)
  void* K; void* VT; long long sb, sh; int S;                      // caches as in AttnArgs; row r is sequence r
  int H, Hkv, hd, R, nsplit;
  int kv_cap;                      // bound on the cached slots of every row (new slot excluded)
  void* o; int ldo;                // o [R][H*hd] (storage type)
  float* part_out;                 // split records as in AttnArgs::part
  bool combine;                    // merge split records into o here (else a staged GEMM does)
  const float* ss; int ss_n, d;    // projection left unscaled: rinv = 1/sqrt(sum of ss[0..ss_n)[r] / d + eps)
  float eps;
  RowMap rm;
  const int* gate; int gate_n;     // launch does nothing unless a gate flag is set (micro steps)
};

// ---------------------------------------------------------------- launchers
typedef hipStream_t Stream;
// tag 0: base-layer launch (distinct kernel name in profiles), 1: any other.
// *nsplit receives the k-split used; above 1 the result is fp32 partials in a.part.
// the split-K partial buffer holds nsplit * M <= PART_ROWS rows of N floats
constexpr int PART_ROWS = 1024;
// returns GEMM_NO_STAGE (nothing launched) when a staged X source does not fit
int launch_gemm(int dtype, int epi, const GemmArgs& a, int max_split, Stream s, int tag, int* nsplit);
constexpr int GEMM_NO_STAGE = -2;
// whether launch_gemm would take the staged path for these arguments (nothing launched)
bool gemm_stage_fits(int dtype, int epi, const GemmArgs& a, int max_split);
// the NormOut epilogue (one workgroup per 16-column tile, unsplit): rows up to
// NORM_OUT_MAX_ROWS and at most NORM_OUT_MAX_TILES tiles; the tile count its
// launch uses (-1: does not apply)
constexpr int NORM_OUT_MAX_ROWS = 8, NORM_OUT_MAX_TILES = 256;
constexpr int NORM_OUT_FILL_TILES = 256;  // tiles (unsplit workgroups) that give each of the 256 CUs one
bool gemm_norm_out_fits(int M, int N, int K);
int gemm_norm_out_tiles(int N);
int launch_decide(int dtype, const DecideArgs& d, int ntiles, int M, Stream s);
int skinny_tiles(int N);  // column tiles (argmax partials per row) of a skinny launch over N columns
int launch_split_reduce(int dtype, int epi, const GemmArgs& a, Stream s);
int launch_attn_decode(int dtype, const AttnArgs& a, Stream s);
int launch_attn_prefill(int dtype, const AttnArgs& a, Stream s);
int launch_attn_step(int dtype, const AttnStepArgs& a, Stream s);
int attn_step_max_qkv_split();  // most split-K partials of the projection the step kernel sums

struct RopeArgs {
  const float* qkv; int ldqkv, R;  // [R][(H+2Hkv)hd] fp32 projections
  const float* part; int nsplit;   // or split-K partials [nsplit][R][ldqkv] to sum
  void* q; int ldq;                // out q [R][H*hd]
  void* K; void* VT; long long sb, sh; int S;
  int H, Hkv, hd;
  const float* cos_t; const float* sin_t;  // [max_pos][hd/2]
  int max_pos;
  RowMap rm;
  const int* gate; int gate_n;
};
int launch_rope_append(int dtype, const RopeArgs& a, Stream s);

struct NormArgs {
  float* x; int ldx; int row_stride, row_off;        // input row r = x[(r*row_stride+row_off)*ldx]
  const float* part; int nsplit, pM;                 // pending split-K partials [nsplit][pM][ldx] added to x first
  float* ctx; int ldctx;                             // optional copy of the updated x rows
  const float* g; int d, R; float eps;
  void* out; int ldo;                                 // storage-type output
  float* hid; int ldh;                                // optional fp32 copy of the normed rows
  const int* gate; int gate_n;
  float* ss;                                          // scratch [R][d/256] for the two-phase form, or null
};
int launch_rmsnorm(int dtype, const NormArgs& a, Stream s);
// the norm's first phase alone, for 16..256 rows feeding an XS_NORMW GEMM (-1: does not apply)
int launch_norm_reduce(const NormArgs& a, Stream s);

}  // namespace ham
