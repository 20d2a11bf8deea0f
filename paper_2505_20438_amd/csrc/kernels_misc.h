// Argument blocks and launchers of the small kernels (kernels_misc.hip).
#pragma once
#include "ham_internal.h"

namespace ham {

struct MacroArgs {
  SeqPtrs st;
  int B, d, G;
  const void* E; const void* P;     // token and relative-position embeddings
  float* x; int ldx;                // residual rows [B][d] (bypass rows written here)
  void* emb_in;                     // [B][5][d] embedder GEMM rows (query, tokens 0..3)
  const int* forced_in;             // [B] or null
  const int* teacher_in;            // [B][4] or null
  int* out_tokens; int* out_lens;
  const float* cos_t; const float* sin_t; int max_pos, hd;  // RoPE tables [max_pos][hd/2]
  float* rope_cs;                   // [B][hd]: cos | sin of this step's position, per sequence
};

struct EmbedAttnArgs {
  const float* proj;                // [B*5][3*H*hd]
  const float* part; int nsplit;    // or split-K partials [nsplit][B*5][3*H*hd]
  const int* fused;                 // [B] group size when fused, else 0
  int B, H, d, hd;
  void* out;                        // [B][H*hd] storage type
};

struct PrefillArgs {
  SeqPtrs st;
  int B, P, G;
  const int* pos_in; int ldpos;     // [B][ldpos] positions of the P inputs, or null (0..P-1)
  const int* forced_in; const int* teacher_in;
  int* out_tokens; int* out_lens;
};

struct GatherArgs {
  const int* ids; int R; const void* E; int d, V; float* x; int ldx;
  const float* rows;                // if set: copy fp32 rows [R][d] from here instead of gathering E rows
  int* err;                         // set (bit 2) if an id is out of range
};

struct GenArgs {
  void* dst; int rows, cols; long long row_off; int interleave; int tiled; uint64_t key;
};

void launch_macro_begin(int dtype, const MacroArgs& a, Stream s);
void launch_embed_attn(int dtype, const EmbedAttnArgs& a, Stream s);
void launch_prefill_begin(const PrefillArgs& a, Stream s);
void launch_gather_rows(int dtype, const GatherArgs& a, Stream s);
void launch_copy_row(const float* src, float* dst, int d, Stream s);
// R rows of d fp32 values from src (pitch ld_src floats) to dst (pitch ld_dst); 16-byte aligned rows
int launch_copy_rows(const float* src, long long ld_src, float* dst, long long ld_dst, int R, int d, Stream s);
void launch_gen_normal(int dtype, const GenArgs& a, Stream s);
void launch_fill_f32(float* p, long long n, float v, Stream s);

}  // namespace ham
