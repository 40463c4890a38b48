/*
 * wedlm_model.h -- C ABI of the decoder around the WeDLM decode step on
 * MI355X (gfx950): the layers that produce the window's queries, keys,
 * values and logits.  WeDLM: arXiv 2512.22737.
 *
 * WeDLM-8B keeps the architecture of the Qwen3-8B model it starts from
 * (Sec. 6.1); WeDLM changes the attention pattern (the reordered causal
 * window, Sec. 4.1) and the positions (Eq. 2), not the layers.  Per layer,
 * on the window's rows in the physical order of Eq. (5)/(6):
 *
 *   a = RMSNorm(x) g_attn;  q|k|v = a W_qkv^T;  q, k = RMSNorm per head
 *   (g_q, g_k), then RoPE at the logical position;  x += Attn(q, k, v) W_o^T
 *   (wedlm_window_attn over the layer's cache);  m = RMSNorm(x) g_mlp;
 *   x += (silu(m W_gate^T) * (m W_up^T)) W_down^T
 *
 * and at the end h = RMSNorm(x) g_final, scored by wedlm_lm_head_score.
 * RMSNorm(x) = x / sqrt(mean(x^2) + eps).  The residual stream x is fp32;
 * every matrix operand is bf16 with fp32 accumulation.
 *
 * Conventions of wedlm.h hold: device pointers owned by the caller,
 * contiguous row-major arrays, bf16 as uint16_t bits, nothing allocated or
 * synchronised, every call enqueued on `stream`, WEDLM_E_* codes returned
 * before anything is enqueued.
 */
#ifndef WEDLM_MODEL_H
#define WEDLM_MODEL_H

#include "wedlm.h"

#ifdef __cplusplus
extern "C" {
#endif

/* linear epilogues */
#define WEDLM_EPI_STORE_BF16 0 /* out[t][n]  = bf16(sum)                     */
#define WEDLM_EPI_ADD_F32 1    /* out[t][n] += sum        (fp32 out)         */
#define WEDLM_EPI_SWIGLU 2     /* out[t][n]  = bf16(silu(g) * u)             */

typedef struct {
  int32_t n_layers;   /* L                                                */
  int32_t hidden;     /* Hd, a multiple of 256                            */
  int32_t n_heads;    /* Hq                                               */
  int32_t n_kv_heads; /* Hkv, divides Hq                                  */
  int32_t head_dim;   /* D, 64 or 128; Hq * D a multiple of 64            */
  int32_t inter;      /* MLP inner size I, a multiple of 64               */
  int32_t vocab;      /* V                                                */
  int32_t mask_token; /* embedding row fed for a [M] slot, in [0, V)      */
  double rope_theta;  /* RoPE base (> 1)                                  */
  float rms_eps;      /* RMSNorm epsilon (> 0)                            */
} wedlm_model_config;

/* Weights, bf16, stacked over layers.  Every projection is [out, in] (one
 * row per output feature) in the PACKED layout of wedlm_pack_weights, each
 * layer's matrix packed on its own; embeddings, norms and the output layer
 * are plain row-major. */
typedef struct {
  const uint16_t* embed;      /* [V, Hd]                                  */
  const uint16_t* attn_norm;  /* [L, Hd]                                  */
  const uint16_t* w_qkv;      /* [L, (Hq + 2 Hkv) D, Hd]: q rows, k, v    */
  const uint16_t* q_norm;     /* [L, D]                                   */
  const uint16_t* k_norm;     /* [L, D]                                   */
  const uint16_t* w_o;        /* [L, Hd, Hq D]                            */
  const uint16_t* mlp_norm;   /* [L, Hd]                                  */
  const uint16_t* w_gate_up;  /* [L, 2 I, Hd]: the I gate rows, then up   */
  const uint16_t* w_down;     /* [L, Hd, I]                               */
  const uint16_t* final_norm; /* [Hd]                                     */
  const uint16_t* lm_head;    /* [V, Hd]                                  */
} wedlm_model_weights;

/*
 * wedlm_embed -- x[t] = float(table[tok[t]]); a negative id (a [M] slot) or
 * one >= V reads row mask_token.  tok [M] int32, table [V, Hd] bf16 (Hd a
 * multiple of 8), x [M, Hd] fp32.
 */
int wedlm_embed(const int32_t* tok, int32_t M, int32_t mask_token,
                const uint16_t* table, int32_t V, int32_t Hd, float* x,
                void* stream);

/*
 * wedlm_rmsnorm -- y[t] = bf16(x[t] / sqrt(mean(x[t]^2) + eps) * gain),
 * sum of squares and scaling in fp32.  x [M, Hd] fp32, gain [Hd] bf16,
 * y [M, Hd] bf16; Hd a multiple of 4.
 */
int wedlm_rmsnorm(const float* x, const uint16_t* gain, int32_t M,
                  int32_t Hd, float eps, uint16_t* y, void* stream);

/*
 * wedlm_pack_weights -- lay a row-major weight matrix w [rows, K] out in
 * MFMA tiles, the layout wedlm_linear and the decoder read.  Tile (r, s)
 * holds rows 32r .. 32r+31 and k = 64s .. 64s+63 and is 4 KB at element
 * offset (r * K/64 + s) * 2048; inside it, the 8 values at element
 * (j * 64 + l) * 8 are row 32r + l%32, k = 64s + 32*(l/32) + 8j .. +7
 * (j = 0..3, l = 0..63): lane l's operand of the tile's j-th MFMA.
 * rows a multiple of 32, K a multiple of 64; packed has rows * K elements
 * and must not overlap w.  A one-time conversion of a checkpoint.
 */
int wedlm_pack_weights(const uint16_t* w, int64_t rows, int32_t K,
                       uint16_t* packed, void* stream);

/* Bytes of workspace wedlm_linear needs for this product (0: none, or an
 * invalid shape). */
size_t wedlm_linear_workspace_size(int32_t M, int32_t N, int32_t K,
                                   int32_t epilogue);

/*
 * wedlm_linear -- out = x W^T on bf16 MFMA with fp32 accumulation, summed
 * over K in a fixed order (the result does not depend on the run).
 *   x [M, K] bf16 row-major, w [rows, K] bf16 packed (wedlm_pack_weights),
 *   out [M, ldo] (ldo >= N);
 *   epilogue WEDLM_EPI_STORE_BF16: rows = N, out bf16;
 *            WEDLM_EPI_ADD_F32:    rows = N, out fp32, added in place
 *                                  (the residual stream);
 *            WEDLM_EPI_SWIGLU:     rows = 2N (N gate rows, then N up rows),
 *                                  out bf16 = silu(gate) * up.
 *   N a multiple of 32, K a multiple of 64.  x and out must not overlap.
 * workspace: wedlm_linear_workspace_size() bytes (NULL when that is 0):
 * the fp32 partial products of a residual-add product whose K is split over
 * workgroups, summed into out in split order by a second kernel; its
 * contents on entry do not matter.  Two calls that overlap in time must not
 * share a workspace.
 */
int wedlm_linear(const uint16_t* x, const uint16_t* w, int32_t M, int32_t N,
                 int32_t K, int32_t epilogue, void* out, int32_t ldo,
                 void* workspace, size_t workspace_bytes, void* stream);

/*
 * wedlm_qk_norm_rope -- split one row of q|k|v (the output of W_qkv), RMSNorm
 * each query and key head over its D values (gains q_gain / k_gain [D]),
 * rotate them at pos_ids[t] (Eq. 2; "rotate half" as in wedlm_reorder,
 * angles in fp64) and write
 *   q_out [M, Hq, D], k_out [M, Hkv, D] (bf16), v_out [M, Hkv, D] (copied).
 * qkv [M, (Hq + 2 Hkv) D] bf16, pos_ids [M] int32; D 64 or 128.
 */
int wedlm_qk_norm_rope(const uint16_t* qkv, const uint16_t* q_gain,
                       const uint16_t* k_gain, const int32_t* pos_ids,
                       int32_t M, int32_t Hq, int32_t Hkv, int32_t D,
                       double rope_theta, float eps, uint16_t* q_out,
                       uint16_t* k_out, uint16_t* v_out, void* stream);

/* Bytes of workspace wedlm_model_forward needs (0 for an invalid config). */
size_t wedlm_model_workspace_size(const wedlm_model_config* cfg, int32_t B,
                                  int32_t W, int32_t max_prefix_len);

/*
 * wedlm_model_forward -- Algorithm 1's Forward over the reordered window
 * with the decoder above: wedlm_reorder (indices only), wedlm_embed of the
 * physical-order tokens, L layers (each with wedlm_window_attn over its own
 * cache), the final RMSNorm and wedlm_lm_head_score of EVERY window row.
 *
 * In:
 *   cfg, wt       host structs; the weight pointers are device pointers
 *   win_tok [B, W], win_start [B]       window and committed lengths c
 *   k_cache, v_cache   [L, num_pages, ...] one paged cache per layer, each
 *                      in the layout of wedlm.h
 *   block_table [B, max_pages], max_prefix_len as in wedlm_window_attn
 *   temperature        T of the score (> 0)
 * Out:
 *   perm, pos_ids, tok_phys [B, W], n_obs [B]   (wedlm_reorder)
 *   k_win, v_win [L, B, W, Hkv, D]  every layer's rotated keys and values
 *                                   of the window rows (for the commit)
 *   argmax, entropy, pmax [B, W]    scores of all physical rows (pmax may
 *                                   be NULL); the commit reads the masks'
 *   status [B]                      attention's per-sequence status bits
 * workspace: wedlm_model_workspace_size(cfg, B, W, max_prefix_len) bytes.
 */
int wedlm_model_forward(const wedlm_model_config* cfg,
                        const wedlm_model_weights* wt, const int32_t* win_tok,
                        const int32_t* win_start, int32_t B, int32_t W,
                        const uint16_t* k_cache, const uint16_t* v_cache,
                        int64_t num_pages, const int32_t* block_table,
                        int32_t max_pages, int32_t max_prefix_len,
                        double temperature, int32_t* perm, int32_t* pos_ids,
                        int32_t* tok_phys, int32_t* n_obs, uint16_t* k_win,
                        uint16_t* v_win, int32_t* argmax, float* entropy,
                        float* pmax, int32_t* status, void* workspace,
                        size_t workspace_bytes, void* stream);

/*
 * wedlm_commit_layers -- wedlm_commit_rule for a decoder of n_layers
 * layers: the same commit / selection / refill (Algorithm 1), with the
 * committed rows' keys and values of every layer appended to that layer's
 * cache.  k_win, v_win [n_layers, B, W, Hkv, D] (wedlm_model_forward),
 * k_cache, v_cache [n_layers, num_pages, ...]; other arguments as in
 * wedlm_commit_rule.
 */
int wedlm_commit_layers(int32_t* win_tok, int32_t* win_start,
                        const int32_t* argmax, const float* entropy,
                        double tau, double lambda, const uint16_t* k_win,
                        const uint16_t* v_win, uint16_t* k_cache,
                        uint16_t* v_cache, int64_t num_pages,
                        const int32_t* block_table, int32_t max_pages,
                        int32_t B, int32_t W, int32_t Hkv, int32_t D,
                        int32_t n_layers, int32_t* n_commit,
                        int32_t* committed_tok, int32_t* committed_slot,
                        uint8_t* selected, int32_t* status, int32_t rule,
                        void* stream);

#ifdef __cplusplus
}
#endif

#endif /* WEDLM_MODEL_H */
