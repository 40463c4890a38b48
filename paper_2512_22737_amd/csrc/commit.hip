// Algorithm 1 after the forward: commit the leftmost filled run, extend the
// KV cache with its rows, SelectByEntropy with the distance-adjusted entropy
// of Eq. (11), greedy Sample, and refill the window to W slots.  Two other
// decoding rules share the kernel: block-wise stop-and-wait (Fig. 3,
// Sec. 6.4: the window is the block and is committed only once no mask is
// left, all W slots at once) and one token per step (Sec. 6.2: only the
// smallest adjusted entropy is filled, whatever tau).
//
// One workgroup per sequence.  Wave 0 holds the window, one slot per lane:
//   n         = count of trailing ones of the filled-slot ballot (the leading
//               filled run in logical order; these are physical rows 0..n-1
//               after the stable reordering); under the block rule W when no
//               slot is a mask, else 0;
//   phys(s)   = n_obs + rank of mask s among the masks (Eq. 5/6 inverse);
//   select s  iff (double)H_phys(s) < tau - lambda*(s - s0), evaluated
//               without contraction so it rounds like the scalar reference
//               (s0 = the leftmost mask; never under the one-token rule);
//   fallback  = argmin over masks of (double)H + lambda*(s - s0), leftmost
//               on ties, when nothing passes and a mask exists;
//   the new window is the filled window shifted left by n, masks appended.
// Then every thread of the workgroup copies the n committed K and V rows
// into their cache slots (V transposed, per the page layout), 16 bytes of
// one row and head at a time.
#include "common.h"
#include "wedlm_model.h"

using namespace wedlm;

namespace {

constexpr int kThreads = 256;

struct CommitArgs {
  int32_t* win_tok;
  int32_t* win_start;
  const int32_t* argmax;
  const float* entropy;
  double tau, lam;
  const uint16_t* k_phys;
  const uint16_t* v_phys;
  uint16_t* k_cache;
  uint16_t* v_cache;
  int64_t num_pages;
  const int32_t* bt;
  int max_pages, W, Hkv, D;
  int32_t* n_commit;
  int32_t* committed_tok;
  int32_t* committed_slot;
  uint8_t* selected;
  int32_t* status;
  int rule;               // WEDLM_RULE_*
  int n_layers;           // caches to extend (one per decoder layer)
  int64_t win_lstride;    // elements between layers of k_phys / v_phys
  int64_t cache_lstride;  // elements between layers of k_cache / v_cache
};

#pragma clang fp contract(off)
__device__ __noinline__ double threshold_of(double tau, double lam, int d) {
  return __dsub_rn(tau, __dmul_rn(lam, static_cast<double>(d)));
}
__device__ __noinline__ double adjusted_of(double h, double lam, int d) {
  return __dadd_rn(h, __dmul_rn(lam, static_cast<double>(d)));
}
#pragma clang fp contract(on)

// The committed run of sequence b, computed by wave 0 (lane s = window slot
// s): its length n under the rule, the prefix length c, the cache slot of
// each committed position, and the status bits when a committed position
// has no page inside the cache (then nothing is committed).
struct Run {
  int t;                  // the lane's window token
  bool in, is_mask;
  uint64_t maskb;         // ballot of the mask slots
  int n_o, s0, n, c, slot, bad;
};

__device__ Run committed_run(const CommitArgs& a, int b) {
  Run r;
  const int W = a.W;
  const int s = threadIdx.x;
  r.in = s < W;
  r.t = r.in ? a.win_tok[b * W + s] : 0;
  r.is_mask = r.in && r.t < 0;
  r.maskb = ballot(r.is_mask);
  const uint64_t filledb = ballot(r.in && !r.is_mask);
  r.n_o = __popcll(filledb);
  r.s0 = r.maskb ? __ffsll(static_cast<long long>(r.maskb)) - 1 : W;
  r.n = (a.rule == WEDLM_RULE_BLOCK) ? (r.maskb ? 0 : W) : r.s0;
  r.c = a.win_start[b];
  const int32_t* bt = a.bt + static_cast<int64_t>(b) * a.max_pages;
  // every committed position must have a page inside the cache
  int why = 0;
  r.slot = -1;
  if (s < r.n) {
    const int64_t p = static_cast<int64_t>(r.c) + s;
    const int64_t blk = p / kPage;
    if (r.c < 0 || blk >= a.max_pages) {
      why = WEDLM_SEQ_CAPACITY;
    } else {
      const int id = bt[blk];
      if (id < 0 || id >= a.num_pages) why = WEDLM_SEQ_BAD_PAGE;
      else r.slot = id * kPage + static_cast<int>(p % kPage);
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) why |= __shfl_xor(why, off);
  r.bad = why;
  return r;
}

// KV extend: physical rows 0..n-1 -> positions c..c+n-1 of the caches of
// layers [l0, l1), 16-byte pieces of D/8 bf16 values, spread over the
// workgroup's threads.  K rows are contiguous in both layouts.  For V the
// lanes run over consecutive rows of one (head, 8 values of d), so the
// transposed stores of one page land in contiguous 32-byte rows.  Each
// thread loads up to kAppendBatch pieces of K and of V before storing any,
// so a batch costs one memory round trip.
constexpr int kAppendBatch = 8;

__device__ void append_rows(const CommitArgs& a, int b, int n, int c, int l0,
                            int l1, int h0, int h1) {
  const int W = a.W, D = a.D, Hkv = a.Hkv;
  const int DG = D / 8;
  const int NH = h1 - h0;
  const int32_t* bt = a.bt + static_cast<int64_t>(b) * a.max_pages;
  const int total = n * NH * DG;
  const int all = total * (l1 - l0);
  for (int e0 = 0; e0 < all; e0 += kThreads * kAppendBatch) {
    u16x8_t kv[kAppendBatch], vv[kAppendBatch];
#pragma unroll
    for (int u = 0; u < kAppendBatch; ++u) {
      const int e2 = e0 + u * kThreads + threadIdx.x;
      if (e2 >= all) break;
      const int l = l0 + e2 / total, e = e2 % total;
      const uint16_t* k_phys = a.k_phys + l * a.win_lstride;
      const uint16_t* v_phys = a.v_phys + l * a.win_lstride;
      // K: e = (j, h, dg), dg fastest
      const int dg = e % DG, jh = e / DG;
      kv[u] = *reinterpret_cast<const u16x8_t*>(
          k_phys + ((static_cast<int64_t>(b) * W + jh / NH) * Hkv + h0 +
                    jh % NH) * D + dg * 8);
      // V: e = (h, dg, j), j fastest
      const int j = e % n, hd = e / n;
      vv[u] = *reinterpret_cast<const u16x8_t*>(
          v_phys + ((static_cast<int64_t>(b) * W + j) * Hkv + h0 + hd / DG) *
                       D + (hd % DG) * 8);
    }
#pragma unroll
    for (int u = 0; u < kAppendBatch; ++u) {
      const int e2 = e0 + u * kThreads + threadIdx.x;
      if (e2 >= all) break;
      const int l = l0 + e2 / total, e = e2 % total;
      uint16_t* k_cache = a.k_cache + l * a.cache_lstride;
      uint16_t* v_cache = a.v_cache + l * a.cache_lstride;
      {
        const int dg = e % DG, jh = e / DG;
        const int h = h0 + jh % NH, p = c + jh / NH;
        const int64_t pg = bt[p / kPage];
        *reinterpret_cast<u16x8_t*>(
            k_cache + ((pg * Hkv + h) * kPage + p % kPage) * D + dg * 8) = kv[u];
      }
      {
        const int j = e % n, hd = e / n;
        const int dg = hd % DG, h = h0 + hd / DG, p = c + j;
        const int64_t pg = bt[p / kPage];
        uint16_t* dst =
            v_cache + ((pg * Hkv + h) * D + dg * 8) * kPage + p % kPage;
#pragma unroll
        for (int k = 0; k < 8; ++k) dst[k * kPage] = vv[u][k];
      }
    }
  }
}

// Extends the caches of layer blockIdx.y of sequence blockIdx.x, kv head
// blockIdx.z, before commit_kernel updates the window (it reads the same
// pre-step state and finds the same run).
__global__ __launch_bounds__(kThreads) void kv_append_kernel(CommitArgs a) {
  const int b = blockIdx.x, l = blockIdx.y, h = blockIdx.z;
  __shared__ int s_n, s_c;
  if (threadIdx.x < kWave) {
    const Run r = committed_run(a, b);
    if (threadIdx.x == 0) {
      s_n = r.bad ? 0 : r.n;
      s_c = r.c;
    }
  }
  __syncthreads();
  if (s_n > 0) append_rows(a, b, s_n, s_c, l, l + 1, h, h + 1);
}

__global__ __launch_bounds__(kThreads) void commit_kernel(CommitArgs a) {
  const int b = blockIdx.x;
  const int W = a.W;
  __shared__ int s_n, s_c, s_ok;

  if (threadIdx.x < kWave) {
    const int s = threadIdx.x;
    const Run r = committed_run(a, b);
    const bool in = r.in, is_mask = r.is_mask;
    const int t = r.t, n_o = r.n_o, s0 = r.s0, n = r.n, c = r.c;
    const uint64_t maskb = r.maskb;
    const int slot = r.slot, bad = r.bad;

    if (bad) {
      if (in) {
        a.committed_tok[b * W + s] = -1;
        a.committed_slot[b * W + s] = -1;
        a.selected[b * W + s] = 0;
      }
      if (s == 0) {
        a.n_commit[b] = 0;
        a.status[b] = bad;
        s_ok = 0;
      }
    } else {
      // SelectByEntropy over the mask slots (Eq. 11)
      const int below = __popcll(maskb & ((s == 0) ? 0ull : (~0ull >> (64 - s))));
      const int phys = n_o + below;
      double h = 0.0;
      int tok = 0;
      if (is_mask) {
        h = static_cast<double>(a.entropy[b * W + phys]);
        tok = a.argmax[b * W + phys];
      }
      const int d = s - s0;
      const bool pass = a.rule != WEDLM_RULE_ONE_TOKEN && is_mask &&
                        h < threshold_of(a.tau, a.lam, d);
      const uint64_t passb = ballot(pass);
      bool fb = false;
      if (passb == 0 && maskb != 0) {
        // argmin of (adjusted entropy, slot) over the masks
        double key = is_mask ? adjusted_of(h, a.lam, d) : __builtin_inf();
        if (key != key) key = __builtin_inf();   // a NaN entropy ranks last
        int who = is_mask ? s : 0x7fffffff;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
          const double k2 = __shfl_xor(key, off);
          const int w2 = __shfl_xor(who, off);
          if (k2 < key || (k2 == key && w2 < who)) { key = k2; who = w2; }
        }
        fb = s == who;
      }
      const bool sel = pass || fb;
      const int filled_tok = sel ? tok : (is_mask ? WEDLM_MASK_TOKEN : t);
      const int shifted = __shfl(filled_tok, (s + n) & (kWave - 1));
      if (in) {
        a.selected[b * W + s] = pass ? 1 : (fb ? 2 : 0);
        a.committed_tok[b * W + s] = s < n ? t : -1;
        a.committed_slot[b * W + s] = s < n ? slot : -1;
        a.win_tok[b * W + s] = (s + n < W) ? shifted : WEDLM_MASK_TOKEN;
      }
      if (s == 0) {
        a.win_start[b] = c + n;
        a.n_commit[b] = n;
        a.status[b] = 0;
        s_n = n;
        s_c = c;
        s_ok = 1;
      }
    }
  }
  __syncthreads();
  if (!s_ok) return;

  if (s_n > 0) append_rows(a, b, s_n, s_c, 0, a.n_layers, 0, a.Hkv);
}

}  // namespace

namespace {

int commit_impl(int32_t* win_tok, int32_t* win_start, const int32_t* argmax,
                const float* entropy, double tau, double lambda,
                const uint16_t* k_phys, const uint16_t* v_phys,
                uint16_t* k_cache, uint16_t* v_cache, int64_t num_pages,
                const int32_t* block_table, int32_t max_pages, int32_t B,
                int32_t W, int32_t Hkv, int32_t D, int32_t* n_commit,
                int32_t* committed_tok, int32_t* committed_slot,
                uint8_t* selected, int32_t* status, int32_t rule,
                int32_t n_layers, void* stream) {
  if (!win_tok || !win_start || !argmax || !entropy || !k_phys || !v_phys ||
      !k_cache || !v_cache || !block_table || !n_commit || !committed_tok ||
      !committed_slot || !selected || !status)
    return WEDLM_E_ARG;
  if (tau != tau || lambda != lambda || num_pages < 1 || max_pages < 1)
    return WEDLM_E_ARG;
  if (rule != WEDLM_RULE_STREAMING && rule != WEDLM_RULE_BLOCK &&
      rule != WEDLM_RULE_ONE_TOKEN)
    return WEDLM_E_ARG;
  if (n_layers < 1) return WEDLM_E_SHAPE;
  if (B < 1 || B > (1 << 30) || W < 1 || W > WEDLM_MAX_WINDOW || Hkv < 1 ||
      (D != 64 && D != 128))
    return WEDLM_E_SHAPE;
  if (num_pages * kPage > (1ll << 31)) return WEDLM_E_SHAPE;  // int32 slots
  CommitArgs a{};
  a.win_tok = win_tok; a.win_start = win_start; a.argmax = argmax;
  a.entropy = entropy; a.tau = tau; a.lam = lambda;
  a.k_phys = k_phys; a.v_phys = v_phys; a.k_cache = k_cache; a.v_cache = v_cache;
  a.num_pages = num_pages; a.bt = block_table; a.max_pages = max_pages;
  a.W = W; a.Hkv = Hkv; a.D = D;
  a.n_commit = n_commit; a.committed_tok = committed_tok;
  a.committed_slot = committed_slot; a.selected = selected; a.status = status;
  a.rule = rule;
  a.n_layers = n_layers;
  a.win_lstride = static_cast<int64_t>(B) * W * Hkv * D;
  a.cache_lstride = num_pages * Hkv * kPage * D;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (n_layers > 1 || B >= 4) {
    // one workgroup per (sequence, layer, kv head), before the window
    // changes; the commit kernel then extends no cache.  (With fewer
    // sequences and one layer the commit kernel's own workgroup copies the
    // rows, which saves a launch.)
    if (n_layers > 65535 || Hkv > 65535) return WEDLM_E_SHAPE;
    hipLaunchKernelGGL(kv_append_kernel, dim3(B, n_layers, Hkv),
                       dim3(kThreads), 0, st, a);
    WEDLM_LAUNCH_CHECK();
    a.n_layers = 0;
  }
  hipLaunchKernelGGL(commit_kernel, dim3(B), dim3(kThreads), 0, st, a);
  WEDLM_LAUNCH_CHECK();
  return WEDLM_OK;
}

}  // namespace

extern "C" int wedlm_commit(int32_t* win_tok, int32_t* win_start,
                            const int32_t* argmax, const float* entropy,
                            double tau, double lambda, const uint16_t* k_phys,
                            const uint16_t* v_phys, uint16_t* k_cache,
                            uint16_t* v_cache, int64_t num_pages,
                            const int32_t* block_table, int32_t max_pages,
                            int32_t B, int32_t W, int32_t Hkv, int32_t D,
                            int32_t* n_commit, int32_t* committed_tok,
                            int32_t* committed_slot, uint8_t* selected,
                            int32_t* status, void* stream) {
  return commit_impl(win_tok, win_start, argmax, entropy, tau, lambda, k_phys,
                     v_phys, k_cache, v_cache, num_pages, block_table,
                     max_pages, B, W, Hkv, D, n_commit, committed_tok,
                     committed_slot, selected, status, WEDLM_RULE_STREAMING,
                     1, stream);
}

extern "C" int wedlm_commit_rule(
    int32_t* win_tok, int32_t* win_start, const int32_t* argmax,
    const float* entropy, double tau, double lambda, const uint16_t* k_phys,
    const uint16_t* v_phys, uint16_t* k_cache, uint16_t* v_cache,
    int64_t num_pages, const int32_t* block_table, int32_t max_pages,
    int32_t B, int32_t W, int32_t Hkv, int32_t D, int32_t* n_commit,
    int32_t* committed_tok, int32_t* committed_slot, uint8_t* selected,
    int32_t* status, int32_t rule, void* stream) {
  return commit_impl(win_tok, win_start, argmax, entropy, tau, lambda, k_phys,
                     v_phys, k_cache, v_cache, num_pages, block_table,
                     max_pages, B, W, Hkv, D, n_commit, committed_tok,
                     committed_slot, selected, status, rule, 1, stream);
}

extern "C" int wedlm_commit_layers(
    int32_t* win_tok, int32_t* win_start, const int32_t* argmax,
    const float* entropy, double tau, double lambda, const uint16_t* k_win,
    const uint16_t* v_win, uint16_t* k_cache, uint16_t* v_cache,
    int64_t num_pages, const int32_t* block_table, int32_t max_pages,
    int32_t B, int32_t W, int32_t Hkv, int32_t D, int32_t n_layers,
    int32_t* n_commit, int32_t* committed_tok, int32_t* committed_slot,
    uint8_t* selected, int32_t* status, int32_t rule, void* stream) {
  return commit_impl(win_tok, win_start, argmax, entropy, tau, lambda, k_win,
                     v_win, k_cache, v_cache, num_pages, block_table,
                     max_pages, B, W, Hkv, D, n_commit, committed_tok,
                     committed_slot, selected, status, rule, n_layers,
                     stream);
}
