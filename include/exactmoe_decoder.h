/*
 * exactmoe_decoder.h -- a synthetic decoder around the W4A16 routed-expert
 * layer, for measuring time to first token and decode throughput in the
 * setting of the paper's runtime evaluation (Sec. 4.2, Table 1).
 *
 * The paper runs OLMoE with its routed experts in the W4A16 layer and the
 * router, attention, embeddings, normalization layers and language-model
 * head in BF16 (abstract; Sec. 4.1: 16 sparse layers, 64 experts, top-8,
 * hidden 2048, expert size 1024, SDPA attention, greedy decoding).  It gives
 * no further architecture; this decoder is the textbook pre-norm transformer
 * with those sizes:
 *
 *   x = Embed[token]
 *   per layer l:  n = RMSNorm(x; attn_norm[l]);  [q k v] = n Wqkv[l]^T
 *                 q, k <- rotary positions (rotate-half pairs (i, i + Dh/2),
 *                         angle p * rope_base^(-2i/Dh));  k, v appended to the cache
 *                 x += Wo[l] Attn(q, K, V)       (causal, softmax(q.k / sqrt(Dh)))
 *                 x += MoE_l(RMSNorm(x; moe_norm[l]))   (emoe_moe_forward on caches[l])
 *   logits = W_lm RMSNorm(x_last; final_norm);  next = argmax(logits)
 *
 * Precision: weights and activations bf16 (the residual stream x too);
 * RMSNorm, rotary positions, attention scores, softmax and all sums in fp32;
 * logits fp32.  Conventions of exactmoe.h apply (status codes, caller-owned
 * device buffers, asynchrony on `stream`).
 */
#ifndef EXACTMOE_DECODER_H
#define EXACTMOE_DECODER_H

#include "exactmoe.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Largest KV-cache length (positions) the attention kernel supports. */
#define EMOE_DECODER_MAX_POSITIONS 8192

typedef struct emoe_decoder_dims {
  int32_t n_layers;       /* L sparse decoder layers */
  int32_t n_heads;        /* H attention heads; moe.d_model = H * head_dim */
  int32_t head_dim;       /* Dh: 64, 128 or 256 */
  int32_t vocab;          /* V */
  int32_t max_positions;  /* KV-cache length, <= EMOE_DECODER_MAX_POSITIONS */
  float rope_base;        /* rotary base (e.g. 10000) */
  float rms_eps;          /* RMSNorm epsilon */
  int32_t renormalize;    /* mixture weights renormalized over the top-k (1) or not (0) */
  emoe_dims moe;          /* the routed-expert layer of every decoder layer */
} emoe_decoder_dims;

/* Weights (device bf16, nn.Linear order [out][in]).  Per-layer entries are
 * host arrays of n_layers device pointers; the decoder copies the arrays. */
typedef struct emoe_decoder_weights {
  const uint16_t* embed;               /* [V][d] */
  const uint16_t* lm_head;             /* [V][d] */
  const uint16_t* final_norm;          /* [d] */
  const uint16_t* const* attn_norm;    /* [L] x [d] */
  const uint16_t* const* wqkv;         /* [L] x [3d][d]: rows of Wq, then Wk, then Wv */
  const uint16_t* const* wo;           /* [L] x [d][d] */
  const uint16_t* const* moe_norm;     /* [L] x [d] */
  const uint16_t* const* w_router;     /* [L] x [E][d] */
} emoe_decoder_weights;

typedef struct emoe_decoder emoe_decoder; /* opaque; owned by the library */

/* Bytes of the KV cache: L x 2 x max_positions x H x Dh bf16, laid out
 * [layer][k or v][position][head][dim]. */
size_t emoe_decoder_kv_bytes(const emoe_decoder_dims* dims);
/* Workspace of emoe_decoder_forward for up to max_tokens tokens per call. */
size_t emoe_decoder_workspace_bytes(const emoe_decoder_dims* dims, int32_t max_tokens);

/* Create a decoder over caller-owned weights, one slot cache per layer
 * (host array of n_layers emoe_cache*, each created with dims->moe and a slot
 * bank) and a KV cache (device, emoe_decoder_kv_bytes).  Creates a rocBLAS
 * handle for the dense projections of prompts (more than 4 tokens; decode
 * steps use the library's own GEMV kernel).  EMOE_ESHAPE for unsupported
 * sizes. */
int32_t emoe_decoder_create(const emoe_decoder_dims* dims, const emoe_decoder_weights* weights,
                            emoe_cache* const* caches, void* kv_cache, emoe_decoder** out);
int32_t emoe_decoder_destroy(emoe_decoder* dec);

/* Run T tokens (device int32 [T], ids outside [0, V) are clamped) at
 * positions pos0 .. pos0+T-1 through every layer, appending their keys and
 * values to the KV cache (positions before pos0 must hold earlier tokens'),
 * then the head on the last token: logits (device f32 [V]) and the greedy
 * next token (device int32 [1]; ties to the lower id).  A prompt is one call
 * with pos0 = 0; each decode step is a call with T = 1.  pos0 + T must not
 * exceed max_positions.  stats (nullable) accumulates the MoE layers'
 * counters.  Blocks the host when a layer's cache is not fully resident
 * (emoe_moe_forward's batched expert-id transfer). */
int32_t emoe_decoder_forward(emoe_decoder* dec, const int32_t* tokens, int32_t T, int32_t pos0,
                             float* logits, int32_t* next_token, void* workspace,
                             size_t workspace_bytes, hipStream_t stream, emoe_stats* stats);

#ifdef __cplusplus
}
#endif
#endif /* EXACTMOE_DECODER_H */
