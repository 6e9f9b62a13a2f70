/*
 * spade.h -- C ABI of the speculative-verify library for AMD Instinct MI355X
 * (gfx950).
 *
 * The library implements the cloud side of speculative decoding as SPADE
 * (arXiv 2608.13076) uses it: the verifier M_p scores d draft tokens in one
 * forward pass over d+1 positions (Algorithm 1, the "Cloud" step), accepts
 * the longest verified prefix, replaces the first rejected draft by a draw
 * from p'(x) = norm(max(0, p(x) - q(x))) (Sec. III-C, "Verification
 * criterion"), and updates the context (m <- m + k + 1).  The draft length d
 * is called gamma below.
 *
 * Conventions shared by every call
 * --------------------------------
 * - All device memory belongs to the caller: weights, workspace, KV cache,
 *   inputs and outputs.  The library never allocates or frees device memory;
 *   its handles own small host structures only.
 * - Pointers prefixed d_ are device pointers, h_ are host pointers.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Every
 *   call that takes a stream is asynchronous and stream-ordered unless its
 *   comment says it synchronises.
 * - Calls return SPADE_OK or a negative spade_status and never throw.  On
 *   error nothing is launched and spade_last_error() holds a message (per
 *   thread).
 * - Token ids are int32 in [0, vocab).  Out-of-range ids found on the device
 *   are clamped and flagged in the device error word (spade_get_device_error).
 * - A model and the KV handles built on it must be used from one stream at a
 *   time: calls share the workspace.
 * - Schedule choices that do not change any result (tilings, k-splits,
 *   attention merge, correction slices) and the measurement hooks are
 *   declared in spade_tuning.h.
 */
#ifndef SPADE_H
#define SPADE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct spade_model_s* spade_model;
typedef struct spade_kv_s* spade_kv;

typedef enum {
  SPADE_OK = 0,
  SPADE_EINVAL = -1,       /* bad argument (null pointer, range, shape)        */
  SPADE_ECAPACITY = -2,    /* batch, gamma or KV capacity exceeded             */
  SPADE_EHIP = -3,         /* a HIP runtime call failed                        */
  SPADE_EUNSUPPORTED = -4, /* shape the kernels do not handle (see config)     */
  SPADE_EDEVICE = -5       /* device error word non-zero                       */
} spade_status;

enum { SPADE_GREEDY = 0, SPADE_SAMPLE = 1 };
enum { SPADE_F32 = 0, SPADE_BF16 = 1 };

/* Bits of the device error word. */
enum {
  SPADE_DERR_TOKEN = 1u,    /* a token id was outside [0, vocab); clamped      */
  SPADE_DERR_NAN = 2u,      /* a logit was NaN                                  */
  SPADE_DERR_RESIDUAL = 4u, /* max(0, p - q) had no mass; drew from p instead   */
  SPADE_DERR_NOQ = 8u,      /* a sampling request got no draft_probs; greedy    */
  SPADE_DERR_CAPACITY = 16u, /* a request's length left fewer than gamma + 1 free
                                positions (lens written outside the library's
                                calls); clamped, that call's outputs are invalid */
  SPADE_DERR_COMMIT = 32u   /* spade_kv_commit read an n_accepted outside
                               [0, gamma] of the last verify call; clamped      */
};

/* Weight tensors, row-major [out_features, in_features] unless noted. */
enum {
  SPADE_WQ = 0,     /* [d_model, d_model]                                  */
  SPADE_WK = 1,     /* [d_model, d_model]                                  */
  SPADE_WV = 2,     /* [d_model, d_model]                                  */
  SPADE_WO = 3,     /* [d_model, d_model]                                  */
  SPADE_WGATE = 4,  /* [d_ffn, d_model]                                    */
  SPADE_WUP = 5,    /* [d_ffn, d_model]                                    */
  SPADE_WDOWN = 6,  /* [d_model, d_ffn]                                    */
  SPADE_G_ATTN = 7, /* [d_model] float32 gain of the attention RMSNorm     */
  SPADE_G_FFN = 8,  /* [d_model] float32 gain of the feed-forward RMSNorm  */
  SPADE_EMBED = 9,  /* [vocab, d_model]                                    */
  SPADE_G_FINAL = 10, /* [d_model] float32 gain of the final RMSNorm       */
  SPADE_LM_HEAD = 11  /* [vocab, d_model]                                  */
};

/*
 * The verifier: a pre-RMSNorm decoder (Sec. III-A: embedding, L blocks
 * x_{l+1} = x_l + f_l(x_l) with f_l = attention then feed-forward, LM head,
 * softmax).  Attention is multi-head with rotary position embedding
 * (rotate-half pairing of feature i with i + head_dim/2, angle
 * pos * rope_theta^(-2i/head_dim)), grouped-query when n_kv_heads <
 * n_heads: query head h attends with K/V head h / (n_heads / n_kv_heads),
 * and Wk, Wv have n_kv_heads * head_dim rows; the feed-forward is SwiGLU
 * (silu(h W_gate^T) * (h W_up^T)) W_down^T; RMSNorm(x) = x / sqrt(mean(x^2)
 * + rms_eps) * g; no biases; the LM head is untied.
 *
 * weight_dtype: SPADE_BF16 or SPADE_F32 for every matrix (gains are float32).
 * kv_dtype: storage type of K and V (RoPE is applied before storing).
 * n_kv_heads: 0 (the default: n_heads) or a divisor of n_heads.
 * Supported: head_dim 64 or 128; d_model = n_heads * head_dim; d_model and
 * d_ffn multiples of 256 (bf16 weights) or 128 (f32); any vocab >= 2; at most
 * 15 drafts per request (gamma + 1 <= 16 rows).
 */
typedef struct {
  int32_t n_layers, d_model, n_heads, head_dim, d_ffn, vocab;
  int32_t weight_dtype, kv_dtype;
  float rms_eps, rope_theta;
  int32_t n_kv_heads;
} spade_config;

/* Bytes of the library's weight arena (its own tiled layout; filled by
 * spade_model_load_tensor).  0 if the config is unsupported. */
size_t spade_weight_bytes(const spade_config* cfg);

/* Bytes of the workspace for calls with up to max_batch requests of up to
 * max_gamma drafts each and caches of up to max_len positions.  With a bf16
 * cache and head_dim 128 its activation arrays also hold a prefill forward:
 * min(2048, max_batch * max_len rounded up to 16) rows (about 220 MB at the
 * 7B shape, 363 MB at the 33B shape). */
size_t spade_workspace_bytes(const spade_config* cfg, int max_batch, int max_gamma, int max_len);

/* Bytes of a KV cache holding max_batch requests of max_len positions.  With
 * S = max_len rounded up to a multiple of 256 and KVH the K/V heads, K and V
 * are each [n_layers][max_batch][KVH][S / 256] blocks of head_dim x 256
 * elements.  In a bf16 cache a block holds the B operands of the attention's
 * products in MFMA order, as 1 KB fragments.  K (S = Q K^T): fragments
 * [16][head_dim / 32], fragment (u, s) covering positions 16 u .. + 15 and
 * features 32 s .. + 31 of the block, its 16-byte piece 16 j + i holding
 * features 32 s + 8 j .. + 7 of position 16 u + i.  V (O = P V): fragments
 * [head_dim / 16][8], fragment (t, s) covering features 16 t .. + 15 and
 * positions 32 s .. + 31, its piece 16 j + i holding positions 32 s + 8 j .. + 7
 * of feature 16 t + i.  In a float32 cache a K block is [256][head_dim] (a row
 * per position) and a V block [head_dim][256].  So one wave's fragment load is
 * 1 KB contiguous and one 256-key chunk of K or V one contiguous block.
 * max_len <= 16384. */
size_t spade_kv_bytes(const spade_config* cfg, int max_batch, int max_len);

/* Create a model over caller-owned device buffers: d_weights of
 * spade_weight_bytes() and d_workspace of spade_workspace_bytes() bytes
 * (256-byte aligned).  Synchronises once: writes the RoPE table and clears the
 * workspace's counters and error word on the current device. */
spade_status spade_model_create(const spade_config* cfg, void* d_weights, void* d_workspace,
                                int max_batch, int max_gamma, int max_len, spade_model* out);

/* Copy one tensor (kind = SPADE_WQ .. SPADE_LM_HEAD; layer ignored for the
 * three global tensors) from a row-major device buffer into the arena,
 * re-tiling matrices for the GEMM kernels.  d_src holds bf16 bits (uint16) or
 * float32 as weight_dtype says; gains are always float32.  The source may be
 * freed once the stream has passed this call. */
spade_status spade_model_load_tensor(spade_model m, int kind, int layer, const void* d_src, void* stream);

/* Wrap a caller-owned KV buffer of spade_kv_bytes(cfg, max_batch, max_len)
 * bytes plus device int32 arrays lens[max_batch] (cached positions per
 * request) and pending[max_batch] (the token whose row has not been computed
 * yet: the last prompt token, then each round's correction).  lens and
 * pending start at 0. */
spade_status spade_kv_create(spade_model m, void* d_kv, int max_batch, int max_len,
                             int32_t* d_lens, int32_t* d_pending, spade_kv* out);

/* Set lens[0..B) and pending[0..B) from host arrays (a snapshot restore). */
spade_status spade_kv_set_state(spade_kv kv, int B, const int32_t* h_lens,
                                const int32_t* h_pending, void* stream);

/* Read lens and pending to the host.  Synchronises the stream. */
spade_status spade_kv_get_state(spade_kv kv, int B, int32_t* h_lens, int32_t* h_pending, void* stream);

/* Snapshot lens/pending [B] into caller device buffers (device-to-device) and
 * remember the host-side capacity bound; spade_kv_restore copies them back and
 * restores that bound.  Rows past the restored lengths are stale and get
 * overwritten, so verify -> commit -> restore replays a round exactly. */
spade_status spade_kv_snapshot(spade_kv kv, int B, int32_t* d_lens, int32_t* d_pending, void* stream);
spade_status spade_kv_restore(spade_kv kv, int B, const int32_t* d_lens, const int32_t* d_pending,
                              void* stream);

/* Prefill request b: run d_tokens[0 .. n_tokens-2] through the verifier,
 * appending their K/V at positions lens[b] .. lens[b] + n_tokens - 2, and make
 * d_tokens[n_tokens-1] the pending token (no logits are produced).  This is
 * the context y_{1:m} of Algorithm 1's input. */
spade_status spade_prefill(spade_model m, spade_kv kv, int b, const int32_t* d_tokens,
                           int n_tokens, void* stream);

/*
 * spade_verify -- one cloud verification of gamma drafts for B requests
 * (Algorithm 1, Cloud step; Sec. III-C).
 *
 * For request b the rows [pending_b, d_b,1 .. d_b,gamma] are appended at
 * positions lens[b] .. lens[b] + gamma and run through the verifier in one
 * pass; row i gives p_i = softmax(logits_i / T), the distribution of the token
 * after d_b,i (row gamma: after the last draft).  Then, left to right:
 *   greedy (mode SPADE_GREEDY): d_b,i+1 is accepted iff it is the argmax of
 *     row i (ties: lowest id);
 *   sampling (SPADE_SAMPLE): accepted iff u_b,i * q_b,i(d) < p_b,i(d), in
 *     float32, i.e. with probability min(1, p/q).
 * n_accepted[b] = k, the number accepted before the first rejection (0..gamma).
 * correction[b] = the token that follows the k accepted drafts:
 *   greedy: the argmax of row k;
 *   sampling, k < gamma: a draw from norm(max(0, p_k - q_k));
 *   sampling, k = gamma: a draw from p_gamma (no draft distribution there).
 * Draws use Gumbel-max, argmax_v (log w_v + G_v), with G_v = -log(-log U_v),
 * U_v = ((x_v >> 41) + 0.5) * 2^-23 and x_v output v (0-based) of a SplitMix64
 * stream seeded with the float32 bits of u_b,gamma.
 *
 * d_draft_tokens  int32 [B, gamma] (may be NULL when gamma == 0)
 * d_draft_probs   float32 [B, gamma, vocab] draft distributions q, already
 *                 tempered, used as given; may be NULL if no request samples
 *                 or gamma == 0 (a sampling request without q is verified
 *                 greedily and flags SPADE_DERR_NOQ)
 * d_uniforms      float32 [B, gamma + 1] in [0, 1); NULL if no request samples
 * d_mode          uint8 [B], SPADE_GREEDY or SPADE_SAMPLE
 * temperature     finite and > 0; applied to sampling requests (greedy ignores it)
 * d_n_accepted    int32 [B] out
 * d_correction    int32 [B] out
 * d_logits        float32 [B, gamma + 1, vocab] out (raw logits), or NULL
 *
 * The KV rows of all gamma+1 positions are written but lens is unchanged, so
 * the call can be repeated (idempotent) until spade_kv_commit.  Requires
 * lens[b] + gamma + 1 <= max_len, checked against the host-side upper bound
 * of lens (refreshed from the device, synchronising the stream, when the
 * bound alone fails), and B <= max_batch, gamma <= max_gamma.  A device
 * length the bound did not cover (lens written outside the library) is
 * clamped on the device and flagged SPADE_DERR_CAPACITY.
 */
spade_status spade_verify(spade_model m, spade_kv kv, int B, int gamma,
                          const int32_t* d_draft_tokens, const float* d_draft_probs,
                          const float* d_uniforms, const uint8_t* d_mode, float temperature,
                          int32_t* d_n_accepted, int32_t* d_correction, float* d_logits,
                          void* stream);

/* Prefill of B requests at once: request b caches h_n_tokens[b] - 1 prompt
 * tokens (row b of d_tokens, device int32 [B][ld], ld >= every count) after
 * its current length, and its last prompt token becomes pending -- the same
 * cache contents and state as spade_prefill of each request.  Each forward
 * takes R rows from each of a range of consecutive requests (the GEMMs read
 * each weight once for all rows of the forward): with a bf16 cache and
 * head_dim 128 up to all of a request's prompt, within the workspace's
 * prefill rows (max_batch * max_len rounded up to 16, at most 2048, and at
 * least max_batch * 16); otherwise 16 per request.  A request whose prompt
 * runs out inside a forward contributes placeholder rows, written past its
 * length and only where the cache has room.  Needs lens + h_n_tokens[b] <=
 * max_len (else SPADE_ECAPACITY).  Counts are read from host memory
 * (h_n_tokens) before the call returns. */
spade_status spade_prefill_batch(spade_model m, spade_kv kv, int B, const int32_t* d_tokens, int ld,
                                 const int32_t* h_n_tokens, void* stream);

/* Probabilities softmax(logits / temperature) of `rows` rows of V logits,
 * float32, row-major [rows][V] in and out (device pointers, caller-owned; out
 * may not alias in).  The edge side of Algorithm 1 keeps, for every draft
 * token, the distribution q it was drawn from (Sec. III-C: the acceptance
 * test and the residual need q); with the draft model run through
 * spade_verify with gamma = 0, this turns that call's logits into q.
 * Stream-ordered; SPADE_EINVAL for null pointers, rows < 1, V < 2 or a
 * temperature that is not finite and > 0. */
spade_status spade_softmax(const float* d_logits, int rows, int V, float temperature, float* d_probs,
                           void* stream);

/* Context update after spade_verify (Algorithm 1: append the k accepted
 * tokens and the correction, m <- m + k + 1): lens[b] += n_accepted[b] + 1 and
 * pending[b] = correction[b] for b < B, on the device.  KV rows past the new
 * length are the rolled-back drafts; they are overwritten by the next round.
 * Needs a spade_verify on this cache since the last commit, prefill or state
 * change, covering at least B requests (else SPADE_EINVAL); each n_accepted is
 * clamped to [0, gamma] of that call (SPADE_DERR_COMMIT if it was outside).
 * The host-side upper bound of lens grows by gamma + 1; spade_verify reads the
 * device lengths back (one synchronisation) only when that bound would fail
 * its capacity check, so a long verify -> commit loop needs no host sync. */
spade_status spade_kv_commit(spade_kv kv, int B, const int32_t* d_n_accepted,
                             const int32_t* d_correction, void* stream);

/* Accept/reject and correction alone, from given logits (the last stage of
 * spade_verify).  d_logits float32 [B, gamma + 1, V]; other arguments as in
 * spade_verify.  Needs a model only for its workspace: V <= cfg.vocab. */
spade_status spade_accept_from_logits(spade_model m, int B, int gamma, int V, const float* d_logits,
                                      const int32_t* d_draft_tokens, const float* d_draft_probs,
                                      const float* d_uniforms, const uint8_t* d_mode,
                                      float temperature, int32_t* d_n_accepted,
                                      int32_t* d_correction, void* stream);

/* spade_accept_from_logits for callers that cannot allocate -- code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc --
 * and have no model: the same accept/reject and correction draw (the sliced
 * draw of a call that may sample) with the library's own static device
 * scratch (about 260 KB per device, held until the process ends) instead of
 * a model's workspace.  B <= 64 (else SPADE_ECAPACITY), gamma + 1 <= 16;
 * other arguments as in spade_accept_from_logits.  d_err: device uint32 the
 * call ORs the SPADE_DERR_* bits into (the caller clears it).  Calls no
 * allocating routine.  Calls on one device share its scratch: calls that
 * overlap on one device (different streams, no ordering) race. */
spade_status spade_accept_from_logits_noalloc(int B, int gamma, int V, const float* d_logits,
                                              const int32_t* d_draft_tokens, const float* d_draft_probs,
                                              const float* d_uniforms, const uint8_t* d_mode,
                                              float temperature, int32_t* d_n_accepted,
                                              int32_t* d_correction, uint32_t* d_err, void* stream);

/* Read and clear the device error word.  Synchronises the stream. */
spade_status spade_get_device_error(spade_model m, uint32_t* h_flags, void* stream);

/* Message of the last failed call on this thread ("" if none). */
const char* spade_last_error(void);

void spade_model_destroy(spade_model m);
void spade_kv_destroy(spade_kv kv);

#ifdef __cplusplus
}
#endif

#endif /* SPADE_H */
