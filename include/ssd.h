/*
 * ssd.h -- C ABI of the MI355X (gfx950) implementation of the batched verify
 * step of Spatially Speculative Decoding (SSD).
 *
 * The problem (paper Sec. 3.1, Eq. 1): a frozen decoder-only transformer
 * generates an n x n grid of image-code tokens in raster order after a text
 * prefix, one token per forward pass.  SSD (Sec. 3.3) drafts whole blocks of
 * spatially adjacent tokens -- the rest of the current row in runs of k_h
 * horizontal tokens, then k_v complete rows below -- and verifies a block in
 * ONE backbone forward pass ("Verification as Auto Correction"): every drafted
 * position is corrected independently by (A) greedy argmax, (B) sampling, or
 * (C) acceptance-rejection with the residual distribution, for a fixed number
 * of rounds; a final forward pass commits the corrected block to the KV cache.
 *
 * Conventions for every entry point:
 *  - Return value: SSD_OK (0) or a negative ssd_status.  On error nothing has
 *    been launched and the session/model is unchanged, except SSD_E_DEVICE,
 *    which marks the object unusable.  ssd_last_error() returns a
 *    thread-local message describing the last failure.
 *  - Pointers to arrays may be host or device memory (HIP unified addressing
 *    decides).  Work is enqueued on the object's HIP stream; when any output
 *    array is host memory the call synchronizes the stream before returning,
 *    otherwise it returns without synchronizing.  A session runs on the
 *    stream given to ssd_prefill (the model's if NULL); an image decode on the
 *    stream of its call (the model's if NULL); the model's own stream is the
 *    one given to ssd_init_model and is never replaced.
 *  - The caller owns every array it passes; the library owns the device
 *    weights, the KV cache and all workspaces of a model/session.
 *  - Token ids are vocabulary ids.  Image codes occupy [img_lo, img_hi);
 *    every block (draft) token must lie in that range.  Logits cover only the
 *    image range, in code order.
 *  - Sessions are not thread-safe; distinct sessions on distinct streams are.
 *  - Nothing here allocates pinned host memory or changes stream priorities.
 */
#ifndef SSD_H
#define SSD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SSD_OK = 0,
  SSD_E_INVAL = -1,    /* bad argument (null pointer, shape, id out of range) */
  SSD_E_STATE = -2,    /* call not allowed in the object's current state */
  SSD_E_CAPACITY = -3, /* block would run past the session's max context */
  SSD_E_OOM = -4,      /* device allocation failed */
  SSD_E_DEVICE = -5    /* a HIP call failed, or a single-launch forward pass gave
                          up a bounded dependency wait (reported by the next call
                          that synchronizes); the object is poisoned */
} ssd_status;

typedef enum { SSD_F32 = 0, SSD_BF16 = 1 } ssd_dtype;

/* Correction rules of Sec. 3.3 "Verification as Auto Correction". */
typedef enum {
  SSD_GREEDY = 0,        /* (A) argmax of p_k (ties: lowest id)                  */
  SSD_SAMPLE = 1,        /* (B) a sample of p_k                                  */
  SSD_ACCEPT_REJECT = 2  /* (C) keep t with prob min(p/q,1), else [p-q]_+ sample */
} ssd_rule;

/*
 * Backbone shape.  A standard pre-norm decoder (the paper's backbones are
 * used unmodified, Sec. 3.3): RMSNorm, grouped-query causal attention with
 * rotary embedding over raster positions (rotate-half pairs, base rope_theta),
 * SwiGLU MLP W2(silu(W1 z) * W3 z) (the form Eq. 2 writes out), final RMSNorm
 * and an output layer ("GenHead") restricted to the image codes.
 * n_heads must be a multiple of n_kv_heads; head_dim must be even.
 * bf16 models: d_model, n_heads*head_dim and d_ff must be multiples of 256,
 * d_model at most 8192, head_dim 64 or 128, img_hi-img_lo a multiple of 16.
 * fp32 models: d_model and img_hi-img_lo even.  Other shapes: SSD_E_INVAL.
 */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab;
  int32_t img_lo, img_hi; /* image-code id range [img_lo, img_hi) */
  int32_t dtype;          /* ssd_dtype of weights and KV cache */
  float rms_eps;          /* RMSNorm epsilon (1e-5 in the synthetic models) */
  float rope_theta;       /* rotary base (1e4 in the synthetic models) */
} ssd_model_config;

typedef struct ssd_model ssd_model;
typedef struct ssd_session ssd_session;

/*
 * Upload a model.  `weights` is one packed buffer of elements of the model
 * dtype (bf16 bit patterns as uint16, or float32) holding, in this order and
 * row-major:
 *   tok_emb [vocab][d]
 *   for each layer: attn_norm [d], wq [Hq*D][d], wk [Hkv*D][d], wv [Hkv*D][d],
 *                   wo [d][Hq*D], mlp_norm [d], w1 [d_ff][d] (gate),
 *                   w3 [d_ff][d] (up), w2 [d][d_ff]
 *   final_norm [d], lm_head [vocab][d]
 * (a linear layer W maps y = W x).  The buffer may be host or device memory
 * and is only read during the call; the library repacks the weights into its
 * own device layout.  `stream` is a hipStream_t (NULL = default stream).
 */
ssd_status ssd_init_model(const ssd_model_config* cfg, const void* weights, void* stream, ssd_model** out);

/* Number of elements the packed weight buffer of `cfg` must hold. */
int64_t ssd_weights_numel(const ssd_model_config* cfg);

void ssd_free_model(ssd_model* model);

/*
 * Create a session of B sequences and run the prefix ("prefill") pass
 * (Eq. 1's condition c): prefix [B][P] vocabulary ids.  Afterwards every
 * sequence's frontier is f = P and its carry (the logits that score the next
 * position) is the prefix's last logits.  max_ctx bounds P + all committed
 * and drafted positions; max_block bounds the block length K of later
 * verify steps.  The KV cache of max_ctx positions is allocated here.
 */
ssd_status ssd_prefill(ssd_model* model, int32_t B, int32_t P, const int32_t* prefix, int32_t max_ctx,
                       int32_t max_block, void* stream, ssd_session** out);

void ssd_free_session(ssd_session* sess);

typedef struct {
  int32_t rule;        /* ssd_rule */
  int32_t top_k;       /* keep the top_k codes of p and q (<= 0: all); boundary ties keep lower ids */
  double temperature;  /* p = softmax(top_k(logits / temperature)); same warp for q */
  uint64_t seed;       /* key of the counter-based uniforms */
  uint32_t round;      /* verify-round index, part of the uniform's counter */
  int32_t n_fixed;     /* 0 or 1: leading block positions that are already chosen (not verified) */
  int32_t commit;      /* 0: verify-and-correct round; 1: commit pass */
  int32_t truncate;    /* 1: strict greedy verification (exact speculative decoding) */
} ssd_verify_params;

/*
 * One backbone forward pass over a block of K tokens per sequence at
 * positions [f, f+K) of every sequence, under the ordinary causal mask over
 * raster positions (position f+k sees the cache [0, f) and block positions
 * 0..k), followed by the per-position correction (Sec. 3.3).
 *
 * tokens      [B][K] in: current block tokens (drafts or last round's result);
 *             out (verify round): corrected tokens.  Image codes only.
 * ref_logits  [B][K][V_img] or NULL.  Rule (C)'s reference distribution q
 *             (as logits, warped like p).  Non-NULL replaces the stored
 *             reference of every block position; NULL keeps the stored one,
 *             and a position without one uses a point mass at its token.
 * params      see ssd_verify_params.
 * accept_mask [B][K] or NULL: 1 where the position kept its token.
 * accept_count[B] or NULL: accepted positions per sequence.
 * frontier    [B] or NULL: the frontier f after the call.
 * logits_out  [B][K][V_img] or NULL: the pass's logits (position k predicts f+k+1).
 * h_pre_out   [B][K][d] or NULL: last layer hidden state before the final norm.
 *
 * Scoring: block position k is scored by the logits of position k-1, and
 * position 0 by the session's carry.  Positions k < n_fixed are not scored.
 * Verify round (commit = 0): KV slots [f, f+K) are overwritten, f is
 * unchanged; rule (C) rejections store this round's scoring logits as the
 * position's new reference (Sec. 3.3: the previous-round backbone
 * distribution becomes the reference).
 * Commit pass (commit = 1): no correction; the KV slots become final,
 * f += K, the carry becomes the logits of position K-1 and the stored
 * references of the committed positions are dropped.
 * Truncate (truncate = 1, rule (A)): the leading run of positions whose token
 * equals the argmax is accepted, f advances past them (plus the n_fixed
 * positions), and tokens[b][f_new - f_old] receives the argmax at the first
 * mismatch (or after the block): the next block's fixed first token.
 * Errors: SSD_E_INVAL for bad shapes/ids, SSD_E_CAPACITY if f+K > max_ctx,
 * SSD_E_STATE after a device failure.
 * The uniforms of position k are SplitMix64 outputs at the counter
 * (b << 44) | ((f+k) << 20) | (round << 4) | stream, stream 0 = accept test,
 * 1 = sample.
 */
ssd_status ssd_verify_step(ssd_session* sess, int32_t K, int32_t* tokens, const float* ref_logits,
                           const ssd_verify_params* params, uint8_t* accept_mask, int32_t* accept_count,
                           int32_t* frontier, float* logits_out, float* h_pre_out);

/* Copy the current carry logits [B][V_img] (scores of position f; guided
 * sessions: the guided carry of each of the B / 2 images). */
ssd_status ssd_get_carry(ssd_session* sess, float* carry_out);

/*
 * Classifier-free guidance (the paper's backbones decode with it: Table
 * "app_config" lists CFG weights 5.0, 4.0 and 3.0; the mix is that of Ho and
 * Salimans, 2022, applied to logits).  Pairs the session's B sequences
 * (B even): sequence b < B/2 is image b's conditional stream (its prompt),
 * sequence B/2 + b the image's unconditional stream (a null prompt of the same
 * length, prefilled with the session).  From this call on the session
 * decodes B/2 images: ssd_verify_step feeds each image's block to both of its
 * streams and scores every position with the guided logits
 *     l = l_u + weight * (l_c - l_u)
 * (carry included); its tokens, ref_logits, accept_mask, accept_count,
 * frontier and logits_out (guided) arrays have B/2 rows, h_pre_out holds the
 * conditional streams' states, and ssd_get_carry returns the guided carry.
 * Uniforms are keyed by the image index.  A later call changes the weight.
 * Truncate mode is refused on a guided session (SSD_E_INVAL).
 * Errors: SSD_E_INVAL for a NULL session, odd B or a non-finite weight;
 * SSD_E_OOM if the guided-logit buffers cannot be allocated.
 */
ssd_status ssd_session_set_cfg(ssd_session* sess, float weight);

/*
 * SSD image schedule (Sec. 3.3; Sec. 4 "SSD Configuration"; Appendix
 * "Multi-Row Anticipation Ablations"): the prefix prefill, the first image
 * token from the prefill's carry (argmax for rule A, else a sample of the
 * warped carry with uniform stream 2 at round 0), the rest of row 0 in runs
 * of k_h tokens with h_rounds verify rounds each (the first run also carries
 * the first token as a fixed position), then the remaining rows in groups of
 * k_v: b_rounds joint rounds on the group, commit of its leading row, and for
 * each later row of the group i_rounds rounds on the group's uncommitted rows
 * followed by that row's commit.  The verify-round index grows over the whole
 * image.  Passes = 1 + 2*ceil((W-1)/k_h) + sum over groups of m rows of
 * (b + i*(m-1) + m) for h_rounds = 1.
 * cfg = 1 decodes every image with classifier-free guidance of weight
 * cfg_weight (see ssd_session_set_cfg): the prefix then holds 2B prompts, the
 * B conditional ones followed by their B unconditional twins.
 * eol = 1 is the end-of-line layout of backbones that close every image row
 * with one token (their AR step counts are H*(W+1)): row y occupies sequence
 * positions P + y*(W+1) .. P + y*(W+1) + W, the last holding eol_id.  That
 * position rides along with the block that completes its row (the last
 * horizontal run, every row of a vertical group), is never verified or
 * counted, and its logits score the next row's first token; the pass count is
 * unchanged.  With heads (ssd_decode_image_heads) a row end's state is the
 * one that scored the next row's first token.
 * A commit pass followed by a verify round of the block right after it (no
 * head drafting in between) runs, unless separate_commit = 1, as one pass
 * over both blocks: the committed tokens are fixed positions whose KV becomes
 * final, the carry is the logits of the last committed position, and the
 * verify block is scored and corrected in the same pass (the causal mask lets
 * it see the committed block).  Decisions are those of the separate passes;
 * ssd_stats.passes counts the backbone passes actually run.
 * truncate = 1 replaces the schedule by strict greedy verification, the
 * exactness-preserving decode the paper contrasts its own with (Sec. 3.3
 * "Verification as Auto Correction"; it equals greedy AR decoding): blocks of
 * trunc_block raster positions, the first the pending token (the argmax of the
 * carry, already chosen) and the rest the drafts of the next positions; the
 * leading run of drafts equal to the argmax of their scoring logits is
 * accepted, the frontier advances past the pending token and that run, and the
 * argmax at the first mismatch (or after the block) is the next pending token.
 * The pass count then depends on the acceptance.  It needs rule A, cfg = 0,
 * eol = 0 and planted drafts; k_h, h_rounds, k_v, b/i_rounds and
 * separate_commit are ignored.  stats->proposed counts the drafts tested (the
 * accepted ones and the first mismatch of each pass).
 */
typedef struct {
  int32_t grid_h, grid_w;
  int32_t k_h, h_rounds, k_v, b_rounds, i_rounds;
  int32_t rule, top_k;
  double temperature;
  uint64_t seed;
  int32_t cfg;       /* 0: no guidance; 1: classifier-free guidance */
  float cfg_weight;  /* guidance weight w (cfg = 1) */
  int32_t eol;       /* 0: rows follow each other; 1: every row ends with the token eol_id */
  int32_t eol_id;    /* end-of-line vocabulary id (eol = 1) */
  int32_t separate_commit; /* 0: a commit pass and the verify round right after it run as one pass;
                              1: one backbone pass per plan step */
  int32_t truncate;        /* 0: the schedule above; 1: strict greedy verification decode */
  int32_t trunc_block;     /* truncate = 1: positions per block (pending token + drafts), >= 2 */
} ssd_schedule;

typedef struct {
  int64_t passes;        /* backbone forward passes, prefill included */
  int64_t verify_rounds; /* verify passes */
  int64_t accepted;      /* accepted positions summed over verify rounds and sequences */
  int64_t proposed;      /* verified positions summed over verify rounds and sequences */
  /* the same split by the round of the block: index j counts the (j+1)-th verify
     round since the positions were drafted (rounds past the 8th are added to
     index 7); index 0 is round-1 acceptance.  Strict decodes count under 0. */
  int64_t accepted_round[8];
  int64_t proposed_round[8];
  int64_t wall_ns;       /* host wall-clock time of the call, nanoseconds */
} ssd_stats;

/*
 * Decode B images: prefix [B][P] ([2B][P] with cfg = 1); drafts [B][H][W] image-code ids used as
 * the draft of every position (planted drafts); draft_logits
 * [B][H][W][V_img] or NULL (rule C reference for a position's first round,
 * NULL = point masses); out_tokens [B][H][W].  stats may be NULL.
 * The model keeps one decode workspace (KV cache for P + H*W positions)
 * between calls with the same shape.
 */
ssd_status ssd_decode_image(ssd_model* model, const ssd_schedule* sched, int32_t B, int32_t P,
                            const int32_t* prefix, const int32_t* drafts, const float* draft_logits,
                            int32_t* out_tokens, ssd_stats* stats, void* stream);

/*
 * Planted drafts at a controlled acceptance (a measurement input; the paper's
 * trained heads are not available).  Runs the decode ssd_decode_image would
 * run for `sched` (the same passes and decisions, the strict decode too) with
 * drafts made on the fly: right before the first verify round of a block, its
 * draft positions are filled left to right, position x with a_x, the greedy
 * argmax (lowest code among equal maxima) of the backbone's logits for x given
 * the committed context and the block's earlier drafts, if keep[b][x] != 0,
 * else with the code repl[b][x] + (repl[b][x] >= a_x), a uniformly drawn code
 * other than a_x when repl is uniform over [0, V_img - 1).  Each a_x comes
 * from a single-position forward pass whose KV slot the verify pass then
 * overwrites; under rule A a kept draft is accepted in its first round unless
 * the block pass, which adds in another order, moves the argmax (near-equal
 * top logits only).  Strict decodes plant only what a pass tests: the leading
 * kept drafts and the first replaced one.
 * keep [B][H][W] uint8, repl [B][H][W] int32 (image-code indices, not ids),
 * host or device.  drafts_out [B][H][W] receives the planted draft of every
 * position (vocabulary ids; positions never drafted hold repl + img_lo): given
 * to ssd_decode_image as `drafts` with the same schedule it reproduces this
 * call's tokens, counts and passes.  out_tokens and stats as for
 * ssd_decode_image; stats->passes leaves the planting passes out.  Guidance,
 * the end-of-line layout and draft logits are not available here
 * (SSD_E_INVAL); other errors as for ssd_decode_image.
 */
ssd_status ssd_plant_image(ssd_model* model, const ssd_schedule* sched, int32_t B, int32_t P,
                           const int32_t* prefix, const uint8_t* keep, const int32_t* repl, int32_t* drafts_out,
                           int32_t* out_tokens, ssd_stats* stats, void* stream);

/*
 * Measurement hook.  enable = 1 starts recording a HIP event pair around every
 * projection-GEMM and attention launch of the model's forward passes, and
 * around every single-launch forward pass (on the stream they run on);
 * enable = 0 stops.  ssd_profile_read fills, per class c = 0 QKV, 1 O-proj,
 * 2 gate/up, 3 down, 4 LM head, 5 attention, 6 whole forward pass in one
 * launch, 7 the launches of classes 0-4 that ran on the tiled (many-row) GEMM
 * kernel (counted in their own class too): ms[c] = summed kernel time,
 * launches[c] = launch count, bytes[c] = algorithmic HBM bytes of those
 * launches (weights + activations read + outputs written, KV read/written for
 * attention; class 6: the sum of classes 0-5 for that pass) and flops[c] =
 * algorithmic flops (2 M N K per GEMM; 4 D per query head and visible key for
 * attention); reset = 1 clears the totals afterwards.  Arrays have 8 entries;
 * any may be NULL.  Synchronizes the model's stream and every recorded launch.
 */
ssd_status ssd_profile(ssd_model* model, int32_t enable);
ssd_status ssd_profile_read(ssd_model* model, double* ms, int64_t* launches, double* bytes, double* flops,
                            int32_t reset);

/*
 * Spatial draft head f_phi (Sec. 3.3 "Draft Prediction in Latent Space",
 * Eq. 2).  From the last layer's pre-norm hidden state h of a decoded
 * position and the embedding e of its token, a head predicts the state at
 * its spatial offset,
 *     u = W0 [h; e],   h_hat = u + W2 (silu(W1 n) * (W3 n)),   n = g * u / rms(u),
 * and drafts argmax_v GenHead(RMSNorm(h_hat))_v through the backbone's own
 * final norm and output layer (image codes only).  A vertical head drafts a
 * whole row below a committed row in one call (rows are independent).
 *
 * ssd_draft_head_numel: element count of the packed head weights for the
 *   model's d_model and the head's inner size m (-1 if invalid).
 * ssd_draft_head_init: weights in the model's dtype (bf16 bit patterns as
 *   uint16, or float32), host or device, packed W0 [d][2d] (columns: h then
 *   e), g [d], W1 [m][d], W3 [m][d], W2 [d][m]; m a positive multiple of 256;
 *   max_rows >= 1 bounds R of every run.  The head is tied to the model (free it first) and runs
 *   on the model's stream.
 * ssd_draft_head_run: h [R][d] fp32 pre-norm states (e.g. the h_pre_out of a
 *   commit pass), tokens [R] vocabulary ids of the same positions; writes
 *   drafts [R] (absolute image-code ids: lowest id among equal maxima) and,
 *   if logits_out != NULL, the draft logits [R][V_img] fp32 (their softmax is
 *   the draft distribution q of rule C).  Synchronizes when an output is in
 *   host memory.  Errors as for the other entry points (SSD_E_DEVICE poisons
 *   the head).
 */
typedef struct ssd_draft_head ssd_draft_head;
int64_t ssd_draft_head_numel(const ssd_model* model, int32_t m);
ssd_status ssd_draft_head_init(ssd_model* model, int32_t m, const void* weights, int32_t max_rows,
                               ssd_draft_head** out);
ssd_status ssd_draft_head_run(ssd_draft_head* head, int32_t R, const float* h, const int32_t* tokens,
                              int32_t* drafts, float* logits_out);
void ssd_free_draft_head(ssd_draft_head* head);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * computation and results as ssd_draft_head_run, with the run's workspace
 * (staged inputs, activations, x^2 partial sums, draft logits, split-K
 * partials and their counters) taken from a static device array of 64 MiB
 * that every GPU the library runs on holds until the process ends, instead of
 * the head's own workspace.  Allocates nothing, never synchronizes, and takes
 * device arrays only (h, tokens, drafts, logits_out; SSD_E_INVAL otherwise).
 * R up to the head's max_rows, as long as its workspace fits the array
 * (about 20 d + 4 m + 4 V_img bytes per row plus the split-K partials of the
 * four GEMMs: a few hundred rows for d = 2048, m = 2d); larger R is refused
 * with SSD_E_INVAL before any launch.  All calls on one GPU share that GPU's array,
 * which keeps the last call's contents (each call clears what must start at
 * zero): calls that overlap on one GPU race, so callers serialize them (one
 * stream, or events between streams).
 */
ssd_status ssd_draft_head_run_noalloc(ssd_draft_head* head, int32_t R, const float* h, const int32_t* tokens,
                                      int32_t* drafts, float* logits_out);

/*
 * Decode B images under the SSD schedule of ssd_decode_image with drafts from
 * spatial heads instead of a planted table (Sec. 3.3: horizontal heads draft
 * the rest of the current row, vertical heads whole rows below).  Before each
 * horizontal run of n tokens after the last chosen token c, horizontal head j
 * (h_heads[j-1], j = 1..n) drafts position c + j; at the start of each group of
 * m rows below a completed row y, vertical head j (v_heads[j-1], j = 1..m)
 * drafts row y + j, one call per head for all W columns of all images.  A
 * head's input for source token t is [h; e(t)], h the pre-norm last-layer
 * state that scored t (the state of the raster position before it: the
 * prompt's last state for the first image token, else a state of the commit
 * pass that cached t's predecessor; conditional streams under guidance).
 * Under rule C the softmax of a position's draft logits is its reference q for
 * its first verify round.  n_h must cover min(k_h, W-1) heads and n_v
 * min(k_v, H-1); horizontal heads need max_rows >= B, vertical heads
 * max_rows >= B*W.  Heads must belong to `model`.  Other arguments, the
 * schedule and the errors are those of ssd_decode_image.
 */
ssd_status ssd_decode_image_heads(ssd_model* model, const ssd_schedule* sched, int32_t B, int32_t P,
                                  const int32_t* prefix, ssd_draft_head* const* h_heads, int32_t n_h,
                                  ssd_draft_head* const* v_heads, int32_t n_v, int32_t* out_tokens,
                                  ssd_stats* stats, void* stream);

/* Thread-local description of the last error (empty string if none). */
const char* ssd_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SSD_H */
