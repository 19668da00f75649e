/*
 * ftts.h -- C ABI of the MI355X (gfx950) IndexTTS-2 inference library.
 *
 * The library runs the autoregressive Text-to-Semantic GPT of IndexTTS-2, a
 * decoder-only GPT-2 style network (Sec. II-A of "Faster IndexTTS-2"), one
 * token per call for a batch of sequences, after a dense prefill of each
 * sequence's conditioning prefix.  The prefix arrives as embeddings rather than
 * token ids and the decoded tokens carry their own position ids, as in the
 * paper's first and third adaptations of the serving engine (Sec. II-C).
 * Linear weights may be bf16 or fp32, or weight-only quantised to W8A16 /
 * W4A16 (Table I caption; Sec. III-B).  It also runs one guided Euler step of
 * the Semantic-to-Mel flow-matching DiT for a batch of utterances
 * (ftts_dit_step, at the end of this file).
 *
 * Conventions for every entry point
 * ---------------------------------
 *  - Pointers are DEVICE pointers unless marked [host].  The caller allocates
 *    and owns every buffer; the library borrows them for the duration of the
 *    call, allocates no device memory and keeps no device state.
 *  - All work is enqueued asynchronously on `stream` (a hipStream_t; NULL is
 *    the default stream).  No call synchronises the host.
 *  - Arguments are validated before anything is enqueued: a call that returns
 *    an error has no side effects.  Errors are negative FTTS_E_* codes, with
 *    a message in ftts_last_error() (thread-local).  A HIP launch failure is
 *    reported as FTTS_E_HIP.  Nothing aborts, exits or throws.
 *  - Device-side data that the host cannot check without synchronising
 *    (token ids, positions, page-table entries, sequence lengths) is
 *    bounds-checked by the kernels: a row whose token, position or page lies
 *    out of range is treated as inactive (no KV write, zero attention output,
 *    sampled id -1) so that no access leaves its buffer.
 *  - Row-major everywhere.  A linear layer y = x W^T + b stores W as [N][K]
 *    (output row n, input column k, k contiguous).
 */
#ifndef FTTS_H
#define FTTS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- error codes ---------------------------------------------------------- */
#define FTTS_OK 0
#define FTTS_E_INVALID_ARG -1 /* null pointer, bad enum, bad count          */
#define FTTS_E_SHAPE -2       /* inconsistent or unsupported dimensions      */
#define FTTS_E_DTYPE -3       /* unknown or mismatched weight dtype          */
#define FTTS_E_ALIGN -4       /* pointer not 16-byte aligned                 */
#define FTTS_E_RANGE -5       /* a host-visible value out of range           */
#define FTTS_E_HIP -6         /* a HIP runtime call or launch failed         */
#define FTTS_E_UNSUPPORTED -7 /* valid but not implemented by this library   */
#define FTTS_E_WORKSPACE -8   /* workspace missing or smaller than needed    */

/* ---- weight storage modes (ftts_config.wdtype) ----------------------------- */
/* FTTS_F32    every tensor fp32, KV cache fp32, activations fp32.
 * FTTS_BF16   every tensor bf16, KV cache bf16.
 * FTTS_W8A16  the four per-layer linears hold int8 codes [N][K] with one bf16
 *             scale per output row [N]; weight = code * scale.  Every other
 *             tensor (embeddings, LayerNorms, biases, LM head) is bf16.
 * FTTS_W4A16  the four per-layer linears hold 4-bit codes packed eight to an
 *             int32 [N][K/8] (column k in bits 4*(k%8) .. 4*(k%8)+3), with one
 *             bf16 scale and one bf16 zero-point per output row and group of
 *             group_size consecutive columns, both [N][K/group_size];
 *             weight = (code - zero) * scale.  Other tensors bf16.
 * In the three 16-bit modes the KV cache is bf16, the residual stream and all
 * accumulation are fp32, and logits are fp32.                               */
#define FTTS_F32 0
#define FTTS_BF16 1
#define FTTS_W8A16 2
#define FTTS_W4A16 3

typedef struct {
    int32_t n_layer;    /* decoder blocks                                        */
    int32_t d_model;    /* residual width; multiple of 128, <= 4096             */
    int32_t n_head;     /* attention heads; n_head * d_head == d_model          */
    int32_t d_head;     /* must be 64                                           */
    int32_t d_ff;       /* MLP width; multiple of 128, <= 16384                 */
    int32_t vocab;      /* semantic vocabulary rows of tok_emb and the LM head  */
    int32_t n_pos;      /* rows of pos_emb                                      */
    int32_t page_size;  /* KV tokens per page; must be 64                       */
    int32_t wdtype;     /* FTTS_F32 / FTTS_BF16 / FTTS_W8A16 / FTTS_W4A16       */
    int32_t group_size; /* W4A16 group along K; must be 128 (ignored otherwise) */
    float ln_eps;       /* LayerNorm epsilon (biased variance)                   */
} ftts_config;

/* One linear layer.  `w` is [N][K] in the mode's storage; `scale` / `zero`
 * are the quantisation parameters (NULL when unused); `bias` is [N] in the
 * activation dtype (fp32 for FTTS_F32, bf16 otherwise). */
typedef struct {
    const void* w;
    const void* scale;
    const void* zero;
    const void* bias;
} ftts_linear;

/* One pre-LayerNorm decoder block (Sec. II-A: GPT-2 family):
 *   x += attn(LN1(x)) W_out^T + b_out ;  x += gelu(LN2(x) W_fc1^T + b_fc1) W_fc2^T + b_fc2
 * qkv.w is [3*d_model][d_model], rows ordered [q | k | v], each block split into
 * n_head heads of d_head consecutive rows; out.w [d][d]; fc1.w [d_ff][d];
 * fc2.w [d][d_ff].  LayerNorm gains/biases are [d] in the activation dtype. */
typedef struct {
    const void* ln1_g;
    const void* ln1_b;
    ftts_linear qkv;
    ftts_linear out;
    const void* ln2_g;
    const void* ln2_b;
    ftts_linear fc1;
    ftts_linear fc2;
} ftts_layer;

/* The whole model.  tok_emb [vocab][d] and pos_emb [n_pos][d] in the activation
 * dtype; layers is a [host] array of n_layer blocks; lnf_g / lnf_b [d]; the LM
 * head [vocab][d] (+ bias [vocab]) is never quantised: fp32 in FTTS_F32 mode,
 * bf16 otherwise.  Every device pointer must be 16-byte aligned. */
typedef struct {
    ftts_config cfg;
    const void* tok_emb;
    const void* pos_emb;
    const ftts_layer* layers;
    const void* lnf_g;
    const void* lnf_b;
    ftts_linear head;
} ftts_weights;

/* Paged KV cache shared by all sequences.  Layout of `base`, in the KV dtype:
 *   [n_layer][n_pages][2 (k, v)][n_head][page_size][d_head]
 * A sequence's token t lives in physical page block_table[b][t / page_size] at
 * slot t % page_size.  Splits of the attention follow logical pages, so results
 * do not depend on which physical pages a sequence holds. */
typedef struct {
    void* base;
    int32_t n_pages;
} ftts_kv_pool;

/* block_table [B][max_pages] int32 physical page ids; seq_lens [B] int32, the
 * number of tokens already cached for each sequence. */
typedef struct {
    const int32_t* block_table;
    const int32_t* seq_lens;
    int32_t max_pages;
} ftts_page_table;

/* Next-token choice.  top_k == 1 is greedy: the largest raw logit, lowest index
 * on ties (temperature and top_p ignored).  Otherwise, in fp32: z = logit / T;
 * keep the top_k largest z (1 <= top_k <= FTTS_MAX_TOP_K; lower index first on
 * ties); weights exp(z - z_max) summed in that order; keep the shortest prefix
 * whose sum reaches top_p times the total; draw by inverse CDF with the
 * caller's uniform u in [0, 1). */
#define FTTS_MAX_TOP_K 64
typedef struct {
    float temperature; /* > 0 */
    int32_t top_k;     /* 1 .. FTTS_MAX_TOP_K */
    float top_p;       /* (0, 1] */
} ftts_sampling;

#define FTTS_MAX_BATCH 64

/* Bytes of device workspace needed by ftts_prefill / ftts_decode_step for up
 * to `max_batch` sequences and, in prefill, up to `max_rows` prefix rows in
 * total.  Returns 0 for an invalid config. */
size_t ftts_workspace_bytes(const ftts_config* cfg, int32_t max_batch, int32_t max_rows);

/* Message for the last error returned on this thread ("" if none). */
const char* ftts_last_error(void);

/* Library version string. */
const char* ftts_version(void);

/* Decode implementation for later ftts_decode_step calls of this process:
 * 0 automatic (the persistent single-launch step when the model and batch
 * qualify -- d_model 1280, 20 heads, d_ff 5120, 256 <= vocab <= 10240, at most
 * 50 layers, 16-bit or quantised weights, batch <= 2, per-layer tensors of each
 * kind at a fixed stride, weight matrices and LayerNorm vectors 16-byte aligned,
 * a 256-CU device on which the occupancy query admits one of its workgroups per
 * CU -- otherwise one kernel per phase).  The persistent step needs its 256
 * workgroups resident together: work launched concurrently on other streams of
 * the same device can delay that until its bounded wait gives up (see
 * ftts_check_workspace).  1 always one kernel per
 * phase, 2 always the persistent step (calls that do not qualify return
 * FTTS_E_UNSUPPORTED). */
int ftts_set_decode_path(int32_t path);

/* Which implementation an ftts_decode_step call on these weights with `batch`
 * sequences would use under the current setting: 1 one kernel per phase, 2 the
 * persistent single-launch step, or a negative FTTS_E_* code if the call would
 * be refused for its weights or batch.  Reads only host memory. */
int ftts_decode_path(const ftts_weights* w, int32_t batch);

/* Synchronises `stream`, then reports FTTS_E_HIP if a persistent decode step on
 * this workspace gave up waiting for one of its inputs (its bounded wait ran
 * out, about a second), FTTS_OK otherwise.  The step that gives up, and every
 * later step on this workspace, writes sampled_out[b] = -1 for every row (so a
 * loop driven by ftts_advance retires every slot) and leaves logits_out
 * unspecified; ftts_prefill clears the condition.  The device-side flag can
 * also be read without a synchronisation: it is the 32-bit word at byte offset
 * 4 of the workspace (0 = no failure). */
int ftts_check_workspace(const void* ws, size_t ws_bytes, void* stream);

/*
 * Weight-only quantisation of one fp32 matrix w [N][K] (Table I caption and
 * Sec. III-B: only the GPT's weights are quantised; activations stay 16-bit).
 * Deterministic and bit-exact:
 *   FTTS_W8A16: per row n, s = bf16(max_k |w| / 127) (s = 1 if that is 0),
 *               code = clamp(rint(w / s), -127, 127) as int8 into codes [N][K];
 *               scales [N] receives the bf16 bits of s; zeros must be NULL.
 *   FTTS_W4A16: per row n and group g of group_size columns,
 *               mn = min(0, min w), mx = max(0, max w),
 *               s = bf16((mx - mn) / 15) (s = 1 if that is 0),
 *               z = clamp(rint(-mn / s), 0, 15),
 *               code = clamp(rint(w / s) + z, 0, 15), packed eight per int32
 *               into codes [N][K/8]; scales and zeros [N][K/group_size] receive
 *               the bf16 bits of s and z.
 * Divisions are IEEE fp32, rint rounds half to even.  w must be finite.
 * K must be a multiple of 16 (W8A16) or of group_size (W4A16, group_size 128).
 */
int ftts_quantize_weights(int32_t wdtype, const float* w, int64_t N, int64_t K,
                          int32_t group_size, void* codes, uint16_t* scales,
                          uint16_t* zeros, void* stream);

/*
 * Dense prefill of B conditioning prefixes (Sec. II-C: conditioning rows enter
 * as embeddings; they receive no position embedding).
 *   prefix_emb  [sum(lens)][d_model] in the activation dtype, sequences packed
 *               in order.
 *   lens        [host] B prefix lengths, each >= 1.
 *   pt, kv      the page table and pool: token t of sequence b is written to
 *               page block_table[b][t / 64], slot t % 64, for every layer.
 *               seq_lens is not read; the caller sets it to lens afterwards.
 *   last_logits [B][vocab] fp32 logits of each sequence's last prefix row, or
 *               NULL to skip the head.
 *   ws          workspace of at least ftts_workspace_bytes(cfg, B, sum(lens)).
 */
int ftts_prefill(const ftts_weights* w, const void* prefix_emb, const int32_t* lens,
                 int32_t B, const ftts_page_table* pt, const ftts_kv_pool* kv,
                 float* last_logits, void* ws, size_t ws_bytes, void* stream);

/*
 * ftts_prefill that assembles the model's own input from ids (the serving
 * adaptations of Sec. II-C): sequence b's prefix is its cond_lens[b]
 * conditioning rows (speaker latents, emotion and speed embeddings -- 34 rows
 * in IndexTTS-2 -- used as given, with no position embedding), followed by its
 * text_lens[b] text tokens, text row i being
 *     tok_emb[vocab + text_ids[i]] + pos_emb[text_pos0 + i]:
 * text and semantic codes share one token table, the text block after the
 * vocab semantic rows (text ids shifted by the semantic vocabulary size), and
 * the text tokens take their own range of the position table starting at
 * text_pos0 (the semantic tokens' range is the caller's choice of `positions`
 * in ftts_decode_step).
 *   cond_emb   [sum cond_lens][d_model] activation dtype (NULL if all are 0).
 *   cond_lens, text_lens  [host][B] int32 >= 0, cond_lens[b] + text_lens[b] >= 1.
 *   text_ids   [sum text_lens] device int32, packed in sequence order; ids
 *              outside [0, text_vocab) read as a zero token row.
 *   text_vocab rows of the text block: tok_emb holds vocab + text_vocab rows.
 *   text_pos0  first position row of the text range; text_pos0 + text_lens[b]
 *              <= n_pos (FTTS_E_RANGE otherwise).
 * Writes KV slots 0 .. cond_lens[b] + text_lens[b] - 1 and, if last_logits is
 * not NULL, the logits of each sequence's last prefix row; every other rule is
 * that of ftts_prefill.
 */
int ftts_prefill_ids(const ftts_weights* w, const void* cond_emb, const int32_t* cond_lens,
                     const int32_t* text_ids, const int32_t* text_lens, int32_t text_vocab,
                     int32_t text_pos0, int32_t B, const ftts_page_table* pt, const ftts_kv_pool* kv,
                     float* last_logits, void* ws, size_t ws_bytes, void* stream);

/*
 * One decode step for B sequences (the per-token generation step of the
 * autoregressive GPT, Sec. II-A / II-C).
 *   tokens      [B] int32 token ids; a negative id marks an inactive slot.
 *   positions   [B] int32 rows of pos_emb (the semantic tokens' own range).
 *   pt          the new token's key/value go to slot seq_lens[b]; attention
 *               covers slots 0 .. seq_lens[b] inclusive.  The caller
 *               increments seq_lens afterwards.
 *   logits_out  [B][vocab] fp32.
 *   sampled_out [B] int32 chosen ids (-1 for inactive slots).
 *   uniforms    [B] fp32 in [0, 1); may be NULL when samp->top_k == 1.
 *   samp        [host] sampling parameters, shared by the batch.
 *   ws          workspace of at least ftts_workspace_bytes(cfg, B, 0); it must
 *               have been zero-filled or passed through ftts_prefill before
 *               the first step (the persistent step keeps its step counter
 *               and exchange buffers there).
 * Safe to capture in a HIP graph: no host synchronisation, no memset, and all
 * per-step inputs are read through device pointers.
 */
int ftts_decode_step(const ftts_weights* w, const int32_t* tokens, const int32_t* positions,
                     const ftts_page_table* pt, const ftts_kv_pool* kv, float* logits_out,
                     int32_t* sampled_out, const float* uniforms, const ftts_sampling* samp,
                     int32_t B, void* ws, size_t ws_bytes, void* stream);

/* Size of the static scratch of ftts_decode_step_static, per GPU. */
#define FTTS_STATIC_SCRATCH_BYTES (12u << 20)

/*
 * ftts_decode_step for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.  It
 * takes no workspace; its scratch (the persistent step's control words and
 * exchange buffers, the per-phase activations and split-K partials of the
 * other decode paths) is a static device array of FTTS_STATIC_SCRATCH_BYTES
 * that each GPU holds, once the first call on it has set it up, until the
 * process ends.  The call allocates nothing and calls no allocating routine.
 * Every argument, the result and the graph-capture safety are those of
 * ftts_decode_step, whose results it reproduces bit for bit.
 *   FTTS_E_WORKSPACE  when the model and batch need more scratch than
 *                     FTTS_STATIC_SCRATCH_BYTES (ftts_workspace_bytes(cfg, B, 0)
 *                     is the need; 8.9 MB for the 24 x 1280 GPT at B = 64).
 * All calls on one GPU share that GPU's array, which keeps the last call's
 * contents: calls that overlap on one GPU (several host threads, or streams
 * whose work can run concurrently) race and must not be issued.  Each call
 * first runs a one-workgroup kernel on `stream` that, after a persistent step
 * gave up waiting (its sampled ids are -1) or every 2^24 steps, clears the
 * array's control words, so a later call starts afresh; no prefill is needed
 * for that (ftts_prefill works on its own workspace as usual).
 */
int ftts_decode_step_static(const ftts_weights* w, const int32_t* tokens, const int32_t* positions,
                            const ftts_page_table* pt, const ftts_kv_pool* kv, float* logits_out,
                            int32_t* sampled_out, const float* uniforms, const ftts_sampling* samp,
                            int32_t B, void* stream);

/*
 * ftts_decode_step that also hands out the step's last-layer hidden state,
 * which the model's mel stage takes as a condition next to the semantic tokens
 * (Sec. II-A; yielding it per step is the fourth serving adaptation of Sec.
 * II-C).
 *   hidden_out  [B][d_model] fp32, 16-byte aligned: row b is LN_f of sequence
 *               b's new last-layer row, i.e. exactly the input the LM head
 *               multiplies (fp32, before any rounding to the activation dtype).
 *               Rows of inactive slots are unspecified.  NULL is allowed and
 *               makes the call identical to ftts_decode_step.
 * Every other argument, the errors and the graph-capture safety are those of
 * ftts_decode_step; FTTS_E_ALIGN if hidden_out is misaligned.
 */
int ftts_decode_step_hidden(const ftts_weights* w, const int32_t* tokens, const int32_t* positions,
                            const ftts_page_table* pt, const ftts_kv_pool* kv, float* logits_out,
                            float* hidden_out, int32_t* sampled_out, const float* uniforms,
                            const ftts_sampling* samp, int32_t B, void* ws, size_t ws_bytes,
                            void* stream);

/*
 * Bookkeeping between two decode steps, done on the device so that a step can
 * be replayed from a captured HIP graph with fixed pointers (the generation loop
 * of the serving engine: one token per sequence per step, Sec. II-C).  For each
 * sequence b with tokens[b] >= 0:
 *   seq_lens[b] += 1 and positions[b] += 1 (the slot and position just used);
 *   if remaining != NULL, remaining[b] -= 1, and when it reaches 0 the sampled id
 *   is replaced by stop_token (in sampled[b] too) and the sequence retires:
 *   tokens[b] = -1;
 *   if retire_on_stop != 0 and sampled[b] == stop_token, the sequence retires
 *   too (the generation loop of Sec. II-C ends an utterance at its stop code);
 *   otherwise tokens[b] = sampled[b];
 *   if history != NULL and *step_counter < max_steps,
 *   history[*step_counter][b] = sampled[b].
 * Sequences with tokens[b] < 0 are left unchanged (history entry -1).  When
 * step_counter != NULL it is incremented once.  All pointers are device int32
 * arrays of B entries (history: [max_steps][B]); 1 <= B <= 1024.
 */
int ftts_advance(int32_t* tokens, int32_t* positions, int32_t* seq_lens, int32_t* sampled,
                 int32_t* remaining, int32_t stop_token, int32_t retire_on_stop, int32_t* history,
                 int32_t* step_counter, int32_t max_steps, int32_t B, void* stream);

/*
 * The sampler of ftts_decode_step on its own: logits [B][V] fp32, uniforms [B]
 * (may be NULL when top_k == 1), sampled_out [B] int32.  No workspace.
 */
int ftts_sample(const float* logits, int32_t B, int32_t V, const ftts_sampling* samp,
                const float* uniforms, int32_t* sampled_out, void* stream);

/* ---- Semantic-to-Mel flow-matching DiT: one guided Euler step ------------------------
 *
 * Sec. II-A: the Semantic-to-Mel module is conditional flow matching with a
 * Diffusion Transformer conditioned on the GPT's hidden states; inference runs an
 * Euler ODE solver with classifier-free guidance over several steps.  Sec. III-A:
 * the DiT has 96M parameters.  The paper gives no block layout; this step reads
 * it as (all weights bf16, biases and LayerNorm parameters bf16, fp32 residual):
 *   e(t) = W_t2 silu(W_t1 s(t) + b_t1) + b_t2, s(t) = [cos(1000 t f_i), sin(1000 t f_i)],
 *          f_i = 10000^(-i / (t_dim/2))
 *   h    = [x | c] W_in^T + b_in + e(t)                  (one row per frame)
 *   h   += Attn(LN1(h)) W_out^T + b_out ; h += gelu(LN2(h) W_fc1^T + b_fc1) W_fc2^T + b_fc2
 *          (ftts_layer blocks; attention over all frames, no mask, no positions)
 *   v(c) = LN_f(h) W_mel^T + b_mel
 *   v    = v(0) + cfg_w (v(c) - v(0)) ;  x' = x + dt v
 */
typedef struct {
    int32_t n_layer, d_model, n_head, d_head, d_ff;
    int32_t n_mel;   /* state width (mel bins) */
    int32_t d_cond;  /* conditioning row width */
    int32_t t_dim;   /* sinusoidal time features (even) */
    float ln_eps;
} ftts_dit_config;

/* in.w [d_model][n_mel + d_cond]; t1.w [d_model][t_dim]; t2.w [d_model][d_model];
 * layers: [host] array of n_layer blocks as in ftts_layer; lnf_g / lnf_b [d_model];
 * mel.w [n_mel][d_model].  Every tensor bf16 (scale / zero unused), 16-byte aligned. */
typedef struct {
    ftts_dit_config cfg;
    ftts_linear in;
    ftts_linear t1;
    ftts_linear t2;
    const ftts_layer* layers;
    const void* lnf_g;
    const void* lnf_b;
    ftts_linear mel;
} ftts_dit_weights;

#define FTTS_DIT_MAX_BATCH 32

/* Workspace bytes for ftts_dit_step over up to max_frames frames in total. */
size_t ftts_dit_workspace_bytes(const ftts_dit_config* cfg, int32_t max_frames);

/* One guided Euler step for a batch of B utterances (Sec. II-B: every stage runs
 * batched over utterances of different lengths), their frames packed one after
 * another instead of padded: utterance b owns frames
 * [sum_{i<b} lens[i], sum_{i<=b} lens[i]) and attends only to its own frames.
 * All utterances share t, dt and cfg_w; both guidance branches run in one pass.
 *   x       [S][n_mel] fp32, the state at time t (S = sum of lens)
 *   cond    [S][d_cond] bf16, conditioning rows (zeroed for the unguided branch)
 *   lens    [host][B] frames per utterance, each >= 1; 1 <= B <= FTTS_DIT_MAX_BATCH
 *   t, dt, cfg_w   time, step, guidance strength (finite host floats)
 *   x_out   [S][n_mel] fp32, x + dt v (may alias x)
 *   v_out   [S][n_mel] fp32, the guided velocity, or NULL
 * Requires d_head == 64, d_model, d_ff and n_mel multiples of 64, n_mel + d_cond a
 * multiple of 64, t_dim even and <= 1024 (FTTS_E_SHAPE / FTTS_E_UNSUPPORTED otherwise).
 * FTTS_E_WORKSPACE if ws_bytes < ftts_dit_workspace_bytes(cfg, S). */
int ftts_dit_step(const ftts_dit_weights* w, const float* x, const void* cond, const int32_t* lens, int32_t B,
                  float t, float dt, float cfg_w, float* x_out, float* v_out, void* ws, size_t ws_bytes,
                  void* stream);

#ifdef __cplusplus
}
#endif
#endif /* FTTS_H */
