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

}  // namespace wedlm
