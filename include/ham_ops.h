/*
 * libham single-kernel entry points, for parity tests and diagnostics.
 *
 * They run one kernel of the decode loop on caller-provided buffers, so a test
 * can check one step at shapes where running the whole model through a CPU
 * reference is too slow (e.g. attention over a 32K-slot cache):
 *  - ham_op_attention_step runs the fused decode-attention step that every
 *    base layer of ham_macro_step launches, with the same split choice for the
 *    same batch and slot bound;
 *  - ham_op_decode_attention runs the attention over an already filled cache
 *    that the micro decoder's first step uses (a different kernel).
 * Same conventions as include/ham.h: C functions, HAM_OK or a negative
 * HAM_E* code, ham_last_error() for the message, "d_" = device pointers, work
 * enqueued on `hip_stream` and valid after it is synchronised.
 *
 * Activation layout ("act rows") of width W: fp32 models store fp32 [W] per row;
 * bf16 models store each value v as the bf16 pair hi = bf16(v), lo = bf16(v - hi)
 * in two planes per row, [hi 0..W) [lo 0..W) (4 bytes per value either way).
 */
#ifndef HAM_OPS_H
#define HAM_OPS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Workspace bytes that ham_op_decode_attention needs for `rows` query rows. */
size_t ham_op_attention_workspace_bytes(int32_t rows, int32_t n_heads, int32_t n_kv_heads, int32_t head_dim);

/* GQA decode attention of one query row per sequence over that sequence's
 * cache (the base-layer attention of a macro-step over the smashed KV cache,
 * Sec. 3.1): out[r, h] = softmax_j(q[r, h] . K[r, h/(H/Hkv), j] / sqrt(hd)) V[...]
 * over slots j < kv_len[r]; rows with enable[r] == 0 (or kv_len 0) get zeros.
 *  dtype        HAM_F32 or HAM_BF16 (cache element type)
 *  d_q          act rows [rows][n_heads*head_dim], RoPE already applied
 *  d_k          [rows][n_kv_heads][slots_cap][head_dim]   (slot-major)
 *  d_vt         [rows][n_kv_heads][slots_cap/32][head_dim][32]   (V in 32-slot
 *               tiles, d-major inside a tile: element (d, slot) at
 *               ((slot/32)*head_dim + d)*32 + slot%32 of its (row, kv head))
 *  d_kv_len     int32 [rows], each <= slots_cap; d_enable int32 [rows]
 *  kv_max       host upper bound of kv_len (chooses the slot split)
 *  d_out        act rows [rows][n_heads*head_dim]
 * head_dim 64 or 128, n_heads/n_kv_heads in 1..4, slots_cap a multiple of 64.
 * HAM_EINVAL on a bad shape, HAM_ENOMEM if the workspace is too small. */
int ham_op_decode_attention(int32_t dtype, int32_t rows, int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                            int32_t slots_cap, const void* d_q, const void* d_k, const void* d_vt,
                            const int32_t* d_kv_len, const int32_t* d_enable, int32_t kv_max, void* d_out,
                            void* d_workspace, size_t workspace_bytes, void* hip_stream);

/* The fused decode-attention step of one base layer of a macro-step (Sec. 3.1:
 * the fused group's single new KV entry is appended, then attention runs over
 * the smashed cache), for one row per sequence:
 *   q = RoPE(q part of qkv[r]), k = RoPE(k part), v = v part, rotate-half RoPE
 *   with the row's factors (pair (i, i + hd/2) rotated by cos[r][i], sin[r][i]);
 *   k and v are rounded to the cache type and written at slot new_slot[r];
 *   out[r, h] = sum_j softmax_j(q_h . K[r, h/(H/Hkv), j] / sqrt(hd)) V[..., j]
 *   over slots j < kv_len[r] (the new slot included; its score uses the
 *   rounded k).
 *  d_qkv        fp32 [rows][(n_heads + 2*n_kv_heads)*head_dim]: all q heads,
 *               then the k heads, then the v heads (before RoPE)
 *  d_cos, d_sin fp32 [rows][head_dim/2]
 *  d_k, d_vt    caches laid out as for ham_op_decode_attention; slot new_slot[r]
 *               is written, slots below it are read
 *  d_kv_len     int32 [rows]: slots after the append; d_new_slot int32 [rows]
 *               must equal kv_len - 1 and be <= kv_cap, else the row writes
 *               nothing, gets zeros and d_err[r] is OR-ed with 8
 *  d_enable     int32 [rows]: 0 = the row writes nothing and gets zeros
 *  kv_cap       host bound on new_slot for every row, < slots_cap; it and `rows`
 *               choose the slot split exactly as a macro-step over `rows`
 *               sequences does (ham_op_attention_step_splits tells how many)
 *  d_err        int32 [rows], in/out (bits are only set)
 *  d_out        act rows [rows][n_heads*head_dim]
 *  d_workspace  at least ham_op_attention_workspace_bytes(rows, ...) bytes
 * rows in 1..64, head_dim 64 or 128, n_heads/n_kv_heads in 1..4, slots_cap a
 * multiple of 64.  HAM_EINVAL on a bad shape or null pointer, HAM_ENOMEM if
 * the workspace is too small. */
int ham_op_attention_step(int32_t dtype, int32_t rows, int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                          int32_t slots_cap, const float* d_qkv, const float* d_cos, const float* d_sin, void* d_k,
                          void* d_vt, const int32_t* d_kv_len, const int32_t* d_new_slot, const int32_t* d_enable,
                          int32_t kv_cap, int32_t* d_err, void* d_out, void* d_workspace, size_t workspace_bytes,
                          void* hip_stream);

/* ham_op_attention_step without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the split records live in a library-owned device
 * array of ham_op_attention_step_noalloc_max_bytes() bytes (4 MiB), one per
 * GPU, kept until the process ends.  The call allocates nothing (no hipMalloc,
 * hipFree or allocating library routine); on its first use on a device it
 * looks up that device's copy of the array (the current device).  Arguments,
 * results and errors as for ham_op_attention_step, plus HAM_ENOMEM when the
 * launch's split records (rows * n_kv_heads * splits * (n_heads/n_kv_heads) *
 * (head_dim + 2) * 4 bytes, none when unsplit) exceed the array.  Every split
 * writes its whole record before the merge reads it, so nothing needs
 * clearing between calls; calls that overlap on one GPU (other streams or
 * host threads) share the array and race. */
int ham_op_attention_step_noalloc(int32_t dtype, int32_t rows, int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                                  int32_t slots_cap, const float* d_qkv, const float* d_cos, const float* d_sin,
                                  void* d_k, void* d_vt, const int32_t* d_kv_len, const int32_t* d_new_slot,
                                  const int32_t* d_enable, int32_t kv_cap, int32_t* d_err, void* d_out,
                                  void* hip_stream);
size_t ham_op_attention_step_noalloc_max_bytes(void);

/* Slot splits (workgroups per row and kv head) that ham_op_attention_step and
 * a macro-step over `rows` sequences use for this slot bound; 0 if invalid. */
int ham_op_attention_step_splits(int32_t dtype, int32_t rows, int32_t n_kv_heads, int32_t head_dim, int32_t kv_cap);

#ifdef __cplusplus
}
#endif
#endif /* HAM_OPS_H */
