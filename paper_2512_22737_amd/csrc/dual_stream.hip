// Dual-stream masking, the training-time attention of Sec. 4.2: a clean
// memory stream (logical positions 0..L-1, Eq. 7/8) followed by the
// prediction stream cut into blocks of B, each block reordered as in
// Sec. 4.1.  Memory tokens attend causally to the memory stream; a token of
// prediction block k attends to the memory positions before block k and,
// causally, to its own reordered block.
//
// That is the decode step's attention once per block: block k of either
// stream is a W = B window over a cached prefix of k*B memory positions
// (for the memory stream the window is its own block, all filled, so the
// result is plain causal attention).  The forward therefore lays the memory
// stream's keys and values out as 16-position pages (the cache layout of
// wedlm.h) and runs the window-attention kernel over the blocks, each block
// table row listing its sequence's pages in order.  Memory block k and
// prediction block k see the same prefix, so with 2B <= WEDLM_MAX_WINDOW
// they run as one window of 2B rows (the kernel's paired mode: each half
// sees the prefix and, causally, only its own block), and every prefix
// tile staged in LDS serves both; larger blocks run one window each.  The
// prefix is read from the pages in HBM/L2; no block-sparse mask is
// materialised.
#include "common.h"
#include "internal.h"
#include "wedlm_train.h"

using namespace wedlm;

namespace {

// memory stream [n_seq, 2L, Hkv, D] rows 0..L-1 -> pages: K [P, Hkv, 16, D],
// V [P, Hkv, D, 16] (P = n_seq * L / 16).  One thread owns 8 consecutive d
// of one head over the 16 positions of a page: it copies those K rows
// (16-byte pieces, neighbouring lanes on neighbouring d) and transposes the
// V rows in registers, so each of its 8 V^T rows is written as 32
// contiguous bytes.
__global__ __launch_bounds__(256) void memory_pages_kernel(
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, int L,
    int Hkv, int D, int64_t n_items, uint16_t* __restrict__ kc,
    uint16_t* __restrict__ vc) {
  static_assert(kPage == 16, "two 8-position halves per page");
  const int64_t it = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (it >= n_items) return;
  const int DG = D / 8;
  const int dg = static_cast<int>(it % DG);
  const int h = static_cast<int>((it / DG) % Hkv);
  const int64_t spg = it / (DG * Hkv);              // sequence * L/16 + page
  const int64_t sq = spg / (L / kPage);
  const int pp = static_cast<int>(spg % (L / kPage));
  const int64_t src0 = ((sq * 2 * L + pp * kPage) * Hkv + h) * D + dg * 8;
  const int64_t rstride = static_cast<int64_t>(Hkv) * D;   // one position
  const int64_t pg = sq * (L / kPage) + pp;
  u16x8_t vv[kPage];
#pragma unroll
  for (int r = 0; r < kPage; ++r)
    vv[r] = *reinterpret_cast<const u16x8_t*>(v + src0 + r * rstride);
#pragma unroll
  for (int r = 0; r < kPage; ++r)
    *reinterpret_cast<u16x8_t*>(kc + ((pg * Hkv + h) * kPage + r) * D + dg * 8) =
        *reinterpret_cast<const u16x8_t*>(k + src0 + r * rstride);
  uint16_t* dst = vc + ((pg * Hkv + h) * D + dg * 8) * kPage;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    u16x8_t lo, hi;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      lo[r] = vv[r][e];
      hi[r] = vv[r + 8][e];
    }
    *reinterpret_cast<u16x8_t*>(dst + e * kPage) = lo;
    *reinterpret_cast<u16x8_t*>(dst + e * kPage + 8) = hi;
  }
}

// entry s = (sequence, stream, block k), or with paired blocks (sequence,
// block k): prefix k*B; block table row: the sequence's L/16 pages in order
__global__ __launch_bounds__(256) void block_meta_kernel(
    int n_blocks, int K, int B, int P, int streams,
    int32_t* __restrict__ prefix, int32_t* __restrict__ bt) {
  const int s = blockIdx.x;
  const int sq = s / (streams * K);
  const int kb = (s % (streams * K)) % K;
  if (threadIdx.x == 0) prefix[s] = kb * B;
  for (int j = threadIdx.x; j < P; j += 256)
    bt[static_cast<int64_t>(s) * P + j] = sq * P + j;
}

struct DsPlan {
  int K, P, n_blocks, max_prefix;
  bool paired;            // memory and prediction block k in one window
  size_t kc, vc, prefix, bt, attn, total;
};

size_t up256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

bool ds_plan(int n_seq, int L, int B, int Hq, int Hkv, int D, DsPlan* p) {
  if (n_seq < 1 || L < 16 || B < 1 || B > WEDLM_MAX_WINDOW || L % B != 0 ||
      L % kPage != 0 || Hkv < 1 || Hq < Hkv || Hq % Hkv != 0 ||
      (D != 64 && D != 128))
    return false;
  const int64_t blocks = 2ll * n_seq * (L / B);
  if (blocks > 65535 || static_cast<int64_t>(n_seq) * L > (1 << 26))
    return false;
  p->K = L / B;
  p->P = L / kPage;
  p->paired = 2 * B <= WEDLM_MAX_WINDOW;
  // block-table rows: one per pair, or one per block
  p->n_blocks = static_cast<int>(p->paired ? blocks / 2 : blocks);
  p->max_prefix = (p->K - 1) * B;
  const size_t kv = static_cast<size_t>(n_seq) * L * Hkv * D * 2;
  size_t off = 0;
  p->kc = off; off += up256(kv);
  p->vc = off; off += up256(kv);
  p->prefix = off; off += up256(static_cast<size_t>(p->n_blocks) * 4);
  p->bt = off; off += up256(static_cast<size_t>(p->n_blocks) * p->P * 4);
  p->attn = off;
  off += up256(p->paired
                   ? window_attn_pairs_workspace_size(n_seq, p->K, B, Hq, Hkv,
                                                      D, p->max_prefix)
                   : wedlm_window_attn_workspace_size(p->n_blocks, B, Hq, Hkv,
                                                      D, p->max_prefix));
  p->total = off;
  return true;
}

}  // namespace

extern "C" size_t wedlm_dual_stream_attn_workspace_size(int32_t n_seq,
                                                        int32_t L,
                                                        int32_t block,
                                                        int32_t Hq,
                                                        int32_t Hkv,
                                                        int32_t D) {
  DsPlan p;
  if (!ds_plan(n_seq, L, block, Hq, Hkv, D, &p)) return 0;
  return p.total;
}

extern "C" int wedlm_dual_stream_attn(const uint16_t* q, const uint16_t* k,
                                      const uint16_t* v, int32_t n_seq,
                                      int32_t L, int32_t block, int32_t Hq,
                                      int32_t Hkv, int32_t D,
                                      float softmax_scale, uint16_t* out,
                                      float* lse, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  if (!q || !k || !v || !out) return WEDLM_E_ARG;
  if (!(softmax_scale > 0.f) || !(softmax_scale < 1e30f)) return WEDLM_E_ARG;
  DsPlan p;
  if (!ds_plan(n_seq, L, block, Hq, Hkv, D, &p)) return WEDLM_E_SHAPE;
  if (!workspace || workspace_bytes < p.total) return WEDLM_E_WORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  uint16_t* kc = reinterpret_cast<uint16_t*>(ws + p.kc);
  uint16_t* vc = reinterpret_cast<uint16_t*>(ws + p.vc);
  int32_t* prefix = reinterpret_cast<int32_t*>(ws + p.prefix);
  int32_t* bt = reinterpret_cast<int32_t*>(ws + p.bt);
  const int64_t items = static_cast<int64_t>(n_seq) * (L / kPage) * Hkv * (D / 8);
  hipLaunchKernelGGL(memory_pages_kernel, dim3((items + 255) / 256), dim3(256),
                     0, st, k, v, L, Hkv, D, items, kc, vc);
  WEDLM_LAUNCH_CHECK();
  hipLaunchKernelGGL(block_meta_kernel, dim3(p.n_blocks), dim3(256), 0, st,
                     p.n_blocks, p.K, block, p.P, p.paired ? 1 : 2, prefix,
                     bt);
  WEDLM_LAUNCH_CHECK();
  if (p.paired)
    return window_attn_pairs(q, k, v, kc, vc,
                             static_cast<int64_t>(n_seq) * p.P, bt, p.P,
                             prefix, n_seq, p.K, block, Hq, Hkv, D,
                             p.max_prefix, softmax_scale, out, lse,
                             ws + p.attn, p.total - p.attn, stream);
  // the blocks in physical order are [n_seq][stream][K] windows of B rows:
  // q, k, v and out viewed as [n_blocks, B, heads, D]
  return wedlm_window_attn(q, k, v, kc, vc,
                           static_cast<int64_t>(n_seq) * p.P, bt, p.P, prefix,
                           p.n_blocks, block, Hq, Hkv, D, p.max_prefix,
                           softmax_scale, out, lse, nullptr, ws + p.attn,
                           p.total - p.attn, stream);
}
