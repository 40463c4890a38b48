/*
 * wedlm_train.h -- C ABI of the training-time attention of WeDLM (arXiv
 * 2512.22737, Sec. 4.2 "Dual-Stream Masking") on MI355X (gfx950): the
 * forward of attention over a clean memory stream and a block-wise
 * reordered prediction stream.
 *
 * Conventions of wedlm.h hold (device pointers owned by the caller, bf16 as
 * uint16_t bits, nothing allocated or synchronised, enqueued on `stream`,
 * WEDLM_E_* codes returned before anything is enqueued).
 */
#ifndef WEDLM_TRAIN_H
#define WEDLM_TRAIN_H

#include "wedlm.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Bytes of workspace wedlm_dual_stream_attn needs (0: unsupported shape). */
size_t wedlm_dual_stream_attn_workspace_size(int32_t n_seq, int32_t L,
                                             int32_t block, int32_t Hq,
                                             int32_t Hkv, int32_t D);

/*
 * wedlm_dual_stream_attn -- attention of Eq. (7)'s input under the block
 * attention pattern of Sec. 4.2, for n_seq sequences of L tokens.
 *
 * Physical rows of one sequence (2L): the memory stream, logical positions
 * 0..L-1 in order; then the prediction stream in L/block blocks of `block`
 * rows, each reordered as in Sec. 4.1 (the block's observed positions
 * first, then its masked ones, each group ascending).  Both streams carry
 * the logical positions 0..L-1 (Eq. 8), so q and k come rotated at the
 * logical position of their row.
 *   memory row at position p      attends to memory rows 0..p;
 *   prediction row of block k     attends to memory positions < k*block and
 *                                 to the rows of its own block up to itself.
 * In:
 *   q [n_seq, 2L, Hq, D], k, v [n_seq, 2L, Hkv, D] bf16 (rows as above),
 *   softmax_scale (usually 1/sqrt(D)); query head h reads kv head
 *   h / (Hq/Hkv).
 * Out:
 *   out [n_seq, 2L, Hq, D] bf16; lse [n_seq, 2L, Hq] fp32 (natural log of
 *   each row's softmax normaliser), or NULL.
 * Limits: block <= 64, L a multiple of block and of 16, D 64 or 128,
 * 2 * n_seq * L / block <= 65535.
 * workspace: wedlm_dual_stream_attn_workspace_size() bytes (the memory
 * stream's keys and values laid out as pages, the block tables, the
 * attention's split partials); its contents on entry do not matter.
 */
int wedlm_dual_stream_attn(const uint16_t* q, const uint16_t* k,
                           const uint16_t* v, int32_t n_seq, int32_t L,
                           int32_t block, int32_t Hq, int32_t Hkv, int32_t D,
                           float softmax_scale, uint16_t* out, float* lse,
                           void* workspace, size_t workspace_bytes,
                           void* stream);

#ifdef __cplusplus
}
#endif

#endif /* WEDLM_TRAIN_H */
