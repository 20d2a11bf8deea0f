/*
 * libham — the HAMburger macro-step decode loop on one AMD MI355X (gfx950).
 *
 * HAMburger (arXiv 2505.20438) stacks a compositional embedder before a base
 * decoder and a micro-step decoder after it (Sec. 3.1, Fig. 2a).  Each macro-step
 * fuses the previous group of up to four tokens into ONE base-model input
 * (Sec. 3.2), runs one base forward that writes ONE KV entry for the whole group
 * (Sec. 3.1; Sec. 3.7 "Token Fusion"), then lets the micro-step decoder emit the
 * next group token by token until a stop test fires (Sec. 3.3); the emitted
 * tokens are final, never verified (Abstract; Sec. 2.2).  Decoding is greedy
 * (Sec. 4.1).  The first token of every group comes from the base LM head and a
 * single-token group bypasses the embedder (Sec. 3.4).
 *
 * Conventions for every entry point:
 *  - All functions are C, never throw, and return HAM_OK (0) or a negative
 *    HAM_E* code; ham_last_error() gives the calling thread's last message.
 *  - "d_" pointers are device memory (HIP), "h_" pointers host memory.  The
 *    caller owns every buffer and the HIP stream; the library keeps non-owning
 *    pointers plus a small host-side handle (freed by ham_destroy).
 *  - ham_prefill and ham_macro_step only enqueue work on the model's stream and
 *    return; their outputs are valid once the stream has been synchronised.
 *  - Token ids are int32 in [0, vocab).  Layouts are row-major.
 */
#ifndef HAM_H
#define HAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HAM_OK 0
#define HAM_EINVAL (-1)  /* bad argument or configuration */
#define HAM_ENOMEM (-2)  /* a caller buffer is smaller than the size query returned */
#define HAM_EHIP (-3)    /* a HIP runtime call failed (message has the HIP error) */
#define HAM_ESTATE (-4)  /* call out of order (e.g. macro-step before prefill) */
#define HAM_ECAP (-5)    /* would exceed the KV / position capacity fixed at init */

#define HAM_F32 0
#define HAM_BF16 1

/* Stop tests (Sec. 3.3 and Sec. 4.4):
 *  HEAD   — a linear stop head on the normed hidden that produced token t_k;
 *           stop after t_k iff its logit s_k > ln((1-c)/c), c = stop_conf
 *           (continue only if 1 - sigmoid(s_k) >= c).  Tested from k = 0.
 *  TOKEN  — the reserved-token variant: at micro index k >= 1, a predicted
 *           stop_id ends the group and is not emitted.
 *  FORCED — the group length is given per step by the caller (benchmarks and
 *           parity tests on random-initialised models); the group ends on the
 *           decision that emits its last token, as with the stop head.
 *  FORCED_TOKEN — FORCED lengths with the reserved-token variant's control
 *           flow (Sec. 4.4): a group of L < max_group tokens ends on one more
 *           micro step, decision k = L (k >= 1), taken as the reserved id and
 *           not emitted.  Emits the same tokens as FORCED; measures the cost of
 *           that extra step against the stop head. */
#define HAM_STOP_HEAD 0
#define HAM_STOP_TOKEN 1
#define HAM_STOP_FORCED 2
#define HAM_STOP_FORCED_TOKEN 3

typedef struct ham_config {
  /* base decoder (Llama family: RMSNorm, RoPE, GQA, SwiGLU; Sec. 4.1) */
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  /* compositional embedder (Sec. 3.2): one multi-head cross-attention layer
   * followed by a linear map (Sec. 4.1); 1 (0 is read as 1) */
  int32_t embed_layers;
  /* micro-step decoder: layers of the base configuration (Sec. 3.3) */
  int32_t micro_layers;
  int32_t max_group;    /* <= 4: micro-step cap (Sec. 3.6, Sec. 4.1) */
  /* base layers whose residual outputs condition the micro decoder (Sec. 3.3,
   * Fig. 2a: outputs of some intermediate base layers plus the final one).
   * n_ctx_layers = 0: C = min(4, n_layers) layers l_i = ceil(i * n_layers / C).
   * Otherwise C = n_ctx_layers in 1..8 and ctx_layers[0..C) are 1-based layer
   * indices, strictly increasing, each in 1..n_layers.  The micro decoder sees
   * them as C prefix rows at local positions 0..C-1. */
  int32_t n_ctx_layers;
  int32_t ctx_layers[8];
  int32_t stop_mode;    /* HAM_STOP_* */
  int32_t stop_id;      /* TOKEN mode reserved id */
  float stop_conf;      /* HEAD mode confidence c in [0, 1] */
  float rope_theta;     /* RoPE base, e.g. 500000 */
  float norm_eps;       /* RMSNorm epsilon, e.g. 1e-5 */
  int32_t dtype;        /* HAM_F32 or HAM_BF16 (weights, KV, GEMM operands) */
  /* capacity, fixed for the life of the model */
  int32_t max_batch;    /* sequences per call, 1..64 */
  int32_t max_prompt;   /* longest prompt */
  int32_t max_steps;    /* macro-steps after prefill (one KV slot per sequence each) */
} ham_config;

/* Per-sequence counters (the "KV entries per output token" metric is
 * gen_slots / tokens; one KV slot per consumed group, Sec. 3.1). */
typedef struct ham_kv_stats_t {
  int32_t kv_len;        /* base KV slots held = prompt_slots + gen_slots */
  int32_t prompt_slots;  /* one per prompt token: prompt tokens are not fused (Fig. 2b) */
  int32_t gen_slots;     /* one per macro-step run for this sequence = groups - 1 */
  int32_t tokens;        /* output tokens emitted (all groups) */
  int32_t groups;        /* groups emitted, including the one from prefill */
  int32_t done;          /* 1 once the token budget is spent */
  int32_t len_hist[5];   /* groups of length 0..4 */
  int32_t device_error;  /* nonzero if a device-side check tripped (bit mask): 1 RoPE position or
                          * KV slot out of range, 2 prompt token id out of range, 4 teacher token
                          * out of range, 8 new KV slot inconsistent with the cache length */
} ham_kv_stats_t;

typedef struct ham_model ham_model;

/* Buffer sizes for a configuration (0 if the configuration is invalid).
 * weights: all parameters, norm gains and RoPE tables;
 * state:   the smashed KV cache of every base layer plus per-sequence counters;
 * workspace: activations, split-K partials and counters of one step. */
size_t ham_weights_bytes(const ham_config* cfg);
size_t ham_state_bytes(const ham_config* cfg);
size_t ham_workspace_bytes(const ham_config* cfg);

/* Validate `cfg`, bind the caller's buffers (each at least the size above,
 * 256-byte aligned) and stream, fill the weights with the seeded N(0, 0.02)
 * initialisation (SplitMix64 counters + Box-Muller, norm gains 1, no biases),
 * build the RoPE tables and clear the state.  Blocks until done.  On success
 * *out is a new handle.  HAM_EINVAL for an invalid configuration or null
 * pointer, HAM_EHIP if a HIP call fails. */
int ham_init_weights(const ham_config* cfg, uint64_t seed, void* d_weights, size_t weights_bytes,
                     void* d_state, size_t state_bytes, void* d_workspace, size_t workspace_bytes,
                     void* hip_stream, ham_model** out);

/* Prefill (Fig. 2b: prompt tokens are not fused, one KV slot each) of `batch`
 * sequences of `prompt_len` tokens, then the first token decision and micro
 * loop, which emit group 1 of every sequence.
 *  d_prompt      int32 [batch][prompt_len]
 *  h_max_new     int32 [batch] output-token budget per sequence (0 = none)
 *  d_forced_lens int32 [batch] group lengths for this step (FORCED and FORCED_TOKEN modes only,
 *                otherwise may be NULL)
 *  d_teacher     int32 [batch][4] or NULL: teacher forcing for parity tests
 *                (FORCED modes only): the group fed back to the model is the
 *                teacher's tokens, while d_out_tokens still reports the
 *                model's own argmax at each position
 *  d_out_tokens  int32 [batch][4] the emitted group, d_out_lens int32 [batch]
 * Resets all per-sequence state.  HAM_EINVAL on bad sizes, HAM_ECAP if
 * prompt_len > max_prompt or batch > max_batch. */
int ham_prefill(ham_model* m, int32_t batch, const int32_t* d_prompt, int32_t prompt_len,
                const int32_t* h_max_new, const int32_t* d_forced_lens, const int32_t* d_teacher,
                int32_t* d_out_tokens, int32_t* d_out_lens);

/* One macro-step for every sequence of the current batch (Sec. 3.1): fuse the
 * previous group (compositional embedder, bypassed for one token), one base
 * forward at the position of the group's last token (Sec. 3.2) writing one KV
 * slot, the first token from the base LM head, then up to max_group-1 micro
 * steps with the on-device stop test.  A sequence whose budget is spent emits
 * nothing (out_len 0) and writes no slot.  Arguments as in ham_prefill.
 * HAM_ESTATE before ham_prefill, HAM_ECAP past max_steps. */
int ham_macro_step(ham_model* m, const int32_t* d_forced_lens, const int32_t* d_teacher,
                   int32_t* d_out_tokens, int32_t* d_out_lens);

/* Test and diagnostics: prefill from caller-given base-model inputs instead of
 * prompt token ids (Sec. 3.1-3.2: a macro-step's base input is one fused vector
 * at the position of its group's last token).  Input t of sequence b is the fp32
 * vector d_embeds [batch][n_inputs][d_model] at RoPE position d_positions int32
 * [batch][n_inputs] (each in [0, max_prompt + 4*(max_steps+1) + 8); checked on
 * device: device_error bit 1).  One causal forward writes KV slots
 * 0..n_inputs-1 (slot order = causal order, whatever the positions), then the
 * first decision and micro loop emit a group; the other arguments are as in
 * ham_prefill.  Fed the recorded inputs of a generation (the prompt tokens'
 * embeddings at 0..P-1, then each macro-step's fused input at its position),
 * this is the full-sequence forward that the incremental macro-steps must
 * reproduce slot for slot.  Later ham_macro_step calls continue from position
 * d_positions[b][n_inputs-1].  HAM_EINVAL on null pointers, HAM_ECAP if
 * n_inputs > max_prompt + max_steps; later macro-steps return HAM_ECAP once
 * the KV slot capacity is spent. */
int ham_prefill_embeds(ham_model* m, int32_t batch, const float* d_embeds, const int32_t* d_positions,
                       int32_t n_inputs, const int32_t* h_max_new, const int32_t* d_forced_lens,
                       const int32_t* d_teacher, int32_t* d_out_tokens, int32_t* d_out_lens);

/* Where the smashed KV cache of base layer `layer` lives in the state buffer
 * (one entry per base input, Sec. 3.1), in the model's storage type, with
 * S = *slots entries of capacity per sequence:
 *   K at *k_offset: [max_batch][n_kv_heads][S][head_dim];
 *   V at *v_offset: 32-entry tiles, element (b, h, s, i) at
 *     ((b*n_kv_heads + h)*(S/32) + s/32)*head_dim*32 + i*32 + s%32.
 * HAM_EINVAL for an invalid configuration or layer. */
int ham_state_info(const ham_config* cfg, int32_t layer, size_t* k_offset, size_t* v_offset, int32_t* slots);

/* Synchronise the stream and copy the counters of each sequence of the current
 * batch into h_out[batch].  HAM_ESTATE before ham_prefill. */
int ham_kv_stats(ham_model* m, ham_kv_stats_t* h_out);

/* Test and diagnostics: when d_buf is non-NULL, every token decision of later
 * calls also writes, for decision k (0..3) of sequence b,
 *   logits  float [4][batch][vocab]   at d_buf
 *   hidden  float [4][batch][d_model] after the logits (normed, before rounding)
 *   stop    float [4][batch]          after the hidden states (stop logits)
 * Requires bytes >= 4*max_batch*(vocab + d_model + 1)*4.  NULL turns it off. */
int ham_set_debug(ham_model* m, void* d_buf, size_t bytes);

/* Number of macro-steps run since the last prefill, or -1. */
int ham_steps_done(const ham_model* m);

/* Save and restore the decode state, so that one prefill can start several
 * decodes (the benchmark times every generation from the same prefilled
 * cache; a server could fork a sequence after a shared prompt).
 * ham_state_save enqueues a device-to-device copy of the whole state buffer
 * (the smashed KV cache and the per-sequence counters, ham_state_bytes bytes)
 * into d_dst and records on the handle the batch, prompt length and macro-step
 * count it belongs to.  ham_state_restore enqueues the copy back from d_src,
 * which must hold what the last ham_state_save of this handle wrote, and
 * resets those host-side fields, so later ham_macro_step calls continue from
 * the saved point.  Both only enqueue work on the model's stream; the caller
 * owns d_dst/d_src and keeps them unchanged in between.  HAM_ESTATE before the
 * first prefill (save) or save (restore), HAM_ENOMEM if bytes <
 * ham_state_bytes. */
int ham_state_save(ham_model* m, void* d_dst, size_t bytes);
int ham_state_restore(ham_model* m, const void* d_src, size_t bytes);

/* Diagnostics: whether ham_macro_step replays its launches from a HIP graph
 * (enable = 1, the default) or launches each kernel on the stream (0).  The
 * graph holds every launch after the step's first kernel, captured once and
 * replayed while the batch, prompt length, output pointers, debug buffer and
 * teacher forcing stay the same; the kernels and their arguments are
 * identical either way (a dependent launch costs about 0.6 us less from a
 * graph).  Timing (ham_profile) always launches on the stream. */
int ham_set_graph(ham_model* m, int enable);

/* Where one generated tensor lives in the weights buffer, by the tensor id of
 * the initialiser (0 E, 1 P, 2..6 A_q A_k A_v A_o A_lin, 7 LM head, 8 stop
 * head, 16 + 8j + t for layer j (base layers first, then micro layers),
 * t = 0..6 Wq Wk Wv Wo Wgate Wup Wdown).  The tensor [rows][cols] is part of a
 * stored matrix of mat_rows rows starting at `offset`: its row r is matrix row
 * row_off + r, except for Wgate/Wup (*interleave 1/2), whose rows are
 * interleaved in blocks of 8 (gate row r at 16*(r/8) + r%8, up row 8 later).
 * Matrices with *tiled = 1 are stored fragment-tiled: element (n, k) of a
 * bf16 matrix with K columns is at
 *   ((n/16 * K/32 + k/32) * 64 + ((k%32)/8) * 16 + n%16) * 8 + k%8
 * (fp32: 16-column fragments of 4 elements per lane); E and P are row-major. */
int ham_tensor_info(const ham_config* cfg, int32_t tensor_id, size_t* offset, int32_t* rows, int32_t* cols,
                    int32_t* row_off, int32_t* mat_rows, int32_t* interleave, int32_t* tiled);

/* Per-kernel-class timing of later calls (diagnostics for the benchmark).
 * While enabled, every launch of the classes below is bracketed by a pair of
 * HIP events on the model's stream and its algorithmic bytes are recorded
 * (weight GEMMs: weights + fp32 activation rows in + fp32 results out;
 * attention: K and V of every visible slot).  Base-layer and k = 0 launches
 * always do their work; micro-step and embedder launches may exit at once when
 * no sequence needs them, so their bytes are upper bounds.
 *   HAM_PROF_QKV, _O, _GU, _DOWN   base-layer projections (decode)
 *   HAM_PROF_MICRO                 micro-decoder layer GEMMs
 *   HAM_PROF_EMBED                 compositional-embedder GEMMs
 *   HAM_PROF_HEAD0                 LM head + argmax + stop test, k = 0
 *   HAM_PROF_HEADK                 the same for micro steps k >= 1
 *   HAM_PROF_ATTN                  split-K decode attention, base layers
 *   HAM_PROF_NORM                  RMSNorm launches (the first kernel of each
 *                                  norm: base and micro layers, decisions);
 *                                  bytes: rows x d x 4 x (pending splits + 3)
 * ham_profile(m, 1) clears the records and starts; ham_profile(m, 0) stops.
 * ham_profile_read synchronises the stream and fills out[kind] for
 * kind < n (launches, summed event time in ms, summed bytes). */
#define HAM_PROF_QKV 0
#define HAM_PROF_O 1
#define HAM_PROF_GU 2
#define HAM_PROF_DOWN 3
#define HAM_PROF_MICRO 4
#define HAM_PROF_EMBED 5
#define HAM_PROF_HEAD0 6
#define HAM_PROF_HEADK 7
#define HAM_PROF_ATTN 8
#define HAM_PROF_NORM 9
#define HAM_PROF_KINDS 10
typedef struct ham_prof_t {
  int32_t launches;
  double ms;
  double bytes;
} ham_prof_t;
int ham_profile(ham_model* m, int enable);
int ham_profile_read(ham_model* m, ham_prof_t* out, int n);

const char* ham_last_error(void);
void ham_destroy(ham_model* m);

#ifdef __cplusplus
}
#endif
#endif /* HAM_H */
