// Library-internal entry points shared between the kernel sources (not part
// of the C ABI; hidden from the shared library's exports).
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace wedlm {

// The window attention of wedlm_window_attn (same arguments, checks and
// errors; no lse) with the output written in the packed MFMA tile layout of
// the projections: element (t, k) of the B*W x Hq*D matrix at
// packed_off(t, k, Hq*D); Hq*D must be a multiple of 64.  Rows of the last
// tile past B*W are not written.
__attribute__((visibility("hidden"))) int window_attn_packed(
    const uint16_t* q_phys, const uint16_t* k_phys, const uint16_t* v_phys,
    const uint16_t* k_cache, const uint16_t* v_cache, int64_t num_pages,
    const int32_t* block_table, int32_t max_pages, const int32_t* prefix_len,
    int32_t B, int32_t W, int32_t Hq, int32_t Hkv, int32_t D,
    int32_t max_prefix_len, float softmax_scale, uint16_t* out_packed,
    int32_t* status, void* workspace, size_t workspace_bytes, void* stream);

// The window attention over paired blocks (dual-stream training attention,
// Sec. 4.2): q, k, v and out are [n_seq][2 streams][blocks][P rows][heads]
// [D]; pair i = (sequence i / blocks, block i % blocks) is one window of
// 2P rows (its stream-0 block, then its stream-1 block) over the prefix of
// prefix_len[i] positions in the paged caches (block-table row i); each
// half sees the prefix and, causally, only its own block.  2P must not
// exceed WEDLM_MAX_WINDOW.  lse [n_seq][2][blocks][P][Hq] or null.  Errors
// as wedlm_window_attn.
__attribute__((visibility("hidden"))) int window_attn_pairs(
    const uint16_t* q, const uint16_t* k, const uint16_t* v,
    const uint16_t* k_cache, const uint16_t* v_cache, int64_t num_pages,
    const int32_t* block_table, int32_t max_pages, const int32_t* prefix_len,
    int32_t n_seq, int32_t blocks, int32_t P, int32_t Hq, int32_t Hkv,
    int32_t D, int32_t max_prefix_len, float softmax_scale, uint16_t* out,
    float* lse, void* workspace, size_t workspace_bytes, void* stream);

// Workspace bytes window_attn_pairs needs (0: unsupported shape).
__attribute__((visibility("hidden"))) size_t window_attn_pairs_workspace_size(
    int32_t n_seq, int32_t blocks, int32_t P, int32_t Hq, int32_t Hkv,
    int32_t D, int32_t max_prefix_len);

}  // namespace wedlm
