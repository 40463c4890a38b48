// Causal GQA attention of the reordered window over the paged prefix cache
// (Sec. 4.1 "Context Awareness under Causal Masking"; Algorithm 1 Forward).
//
// Because the reordering has already moved every filled slot in front of
// every mask, the kernel is a plain causal prefill with a cache offset:
// physical row i sees all c prefix positions and window rows 0..i.  Logical
// positions entered only through RoPE (done by wedlm_reorder).
//
// Work decomposition (one GPU):
//   workgroup = (sequence b, kv head, query block, prefix split)
//   query block = up to 256 rows of the GQA-packed tile: row r = i*G + j is
//                 physical window row i, query head kvh*G + j
//   each wave owns 32 query rows; all waves share 32-key tiles of K and V
//   staged in LDS (double-buffered through registers).
//   S^T = K . Q^T and O^T += V^T . P^T run on v_mfma_f32_32x32x16_bf16:
//   keys are the M dimension of the score tile, so each lane holds 16
//   scores of ONE query column and the row max / row sum need a single
//   cross-half exchange.  The transposed V page layout makes V^T rows
//   contiguous, so both MFMA operands are plain LDS reads.
//   The prefix is split so that the grid fills the 256 CUs; split partials
//   (unnormalised O, running max and sum, log2 domain) are merged by a
//   small combine kernel.  With a single split the main kernel normalises
//   and writes the output itself.
// Roofline: the KV stream, 4 * D * Hkv bytes per prefix position, read once
// per (sequence, kv head, query block); W*G query rows per kv head give an
// arithmetic intensity of W*G flop/byte (256 at W=64, G=4).
#include "common.h"

using namespace wedlm;

namespace {

constexpr int kTileKeys = 32;       // keys per LDS tile (two 16-token pages)
constexpr int kMaxWaves = 8;        // 256 query rows per workgroup
constexpr float kLn2 = 0.69314718055994530942f;

struct AttnArgs {
  const uint16_t* q;      // [B, W, Hq, D]
  const uint16_t* kw;     // [B, W, Hkv, D]
  const uint16_t* vw;     // [B, W, Hkv, D]
  const uint16_t* kc;     // [P, Hkv, 16, D]
  const uint16_t* vc;     // [P, Hkv, D, 16]
  const int32_t* bt;      // [B, max_pages]
  const int32_t* plen;    // [B]
  uint16_t* out;          // [B, W, Hq, D]
  float* lse;             // [B, W, Hq] or null
  int32_t* status;        // [B] or null
  float* ws_o;            // [B, Hkv, rows_pad, nsplit, D]
  float2* ws_ml;          // [B, Hkv, rows_pad, nsplit]
  int64_t num_pages;
  int B, W, Hq, Hkv, G, max_pages, max_prefix, nsplit, split_len, qblocks,
      rows_pad;
  float scale_log2;       // softmax_scale * log2(e)
};

struct Plan {
  int rows, nw, rows_per_wg, qblocks, rows_pad, nsplit, split_len;
  size_t ws_bytes;
};

Plan make_plan(int B, int W, int Hq, int Hkv, int D, int max_prefix) {
  Plan p{};
  const int G = Hq / Hkv;
  p.rows = W * G;
  const int blocks32 = (p.rows + 31) / 32;
  p.nw = blocks32 >= kMaxWaves ? kMaxWaves : (blocks32 >= 4 ? 4 : (blocks32 >= 2 ? 2 : 1));
  p.rows_per_wg = 32 * p.nw;
  p.qblocks = (p.rows + p.rows_per_wg - 1) / p.rows_per_wg;
  p.rows_pad = p.qblocks * p.rows_per_wg;
  const int tiles = (max_prefix + kTileKeys - 1) / kTileKeys;
  const int base = B * Hkv * p.qblocks;
  const int target = 512;  // about two workgroups per CU
  int nsplit = (target + base - 1) / base;
  const int max_split = tiles / 8 > 1 ? tiles / 8 : 1;  // >= 8 tiles each
  if (nsplit > max_split) nsplit = max_split;
  if (nsplit < 1) nsplit = 1;
  int tiles_per = (tiles + nsplit - 1) / nsplit;
  if (tiles_per < 1) tiles_per = 1;
  p.split_len = tiles_per * kTileKeys;
  p.nsplit = (max_prefix + p.split_len - 1) / p.split_len;
  if (p.nsplit < 1) p.nsplit = 1;
  if (p.nsplit == 1) {
    p.ws_bytes = 0;
  } else {
    const size_t n = static_cast<size_t>(B) * Hkv * p.rows_pad * p.nsplit;
    p.ws_bytes = n * D * sizeof(float) + 256 + n * sizeof(float2);
  }
  return p;
}

// LDS row pitches (elements) chosen so the MFMA operand reads are free of
// bank conflicts: 16-byte K reads down 32 rows, 8-byte V^T reads down 32 d.
template <int D>
struct Lds {
  static constexpr int kPitch = D + 8;            // K tile row: one key
  static constexpr int vPitch = kTileKeys + 4;    // V^T tile row: one d
  static constexpr int kElems = kTileKeys * kPitch;
  static constexpr int vElems = D * vPitch;
};

// Sequence validity; bad lengths are reported and the sequence skipped.
__device__ __forceinline__ bool seq_ok(const AttnArgs& a, int b, int& c) {
  c = a.plen[b];
  return c >= 0 && c <= a.max_prefix &&
         static_cast<int64_t>(c) <= static_cast<int64_t>(a.max_pages) * kPage;
}

template <int D, int NW>
struct TileLoader {
  static constexpr int NT = NW * kWave;
  static constexpr int kChunksK = kTileKeys * D / 8;      // 16-byte chunks
  static constexpr int kChunksV = kTileKeys * D / 8;
  static constexpr int kPerThreadK = (kChunksK + NT - 1) / NT;
  static constexpr int kPerThreadV = (kChunksV + NT - 1) / NT;
  u16x8_t rk[kPerThreadK];
  u16x8_t rv[kPerThreadV];

  // Prefix tile: keys p0 .. p0+31, valid below k1.  Returns false and
  // loads zeros if a page id is outside the cache.
  __device__ bool load_prefix(const AttnArgs& a, int b, int kvh, int p0,
                              int k1) {
    const int32_t* bt = a.bt + static_cast<int64_t>(b) * a.max_pages;
    const int pg_idx = p0 / kPage;
    int pg[2];
    bool ok = true;
    for (int h = 0; h < 2; ++h) {
      pg[h] = -1;
      if (p0 + h * kPage < k1) {
        const int id = bt[pg_idx + h];
        if (id >= 0 && id < a.num_pages) pg[h] = id;
        else ok = false;
      }
    }
    const u16x8_t zero = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int u = 0; u < kPerThreadK; ++u) {
      const int ch = threadIdx.x + u * NT;
      rk[u] = zero;
      if (ch < kChunksK) {
        const int key = ch / (D / 8);
        const int col = ch % (D / 8);
        const int h = key / kPage;
        if (pg[h] >= 0 && p0 + key < k1) {
          const uint16_t* src =
              a.kc + ((static_cast<int64_t>(pg[h]) * a.Hkv + kvh) * kPage +
                      (key % kPage)) * D + col * 8;
          rk[u] = *reinterpret_cast<const u16x8_t*>(src);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kPerThreadV; ++u) {
      const int ch = threadIdx.x + u * NT;
      rv[u] = zero;
      if (ch < kChunksV) {
        // chunk = (page half h, d, part): 8 keys of row d of that page
        const int h = ch / (2 * D);
        const int rem = ch % (2 * D);
        const int d = rem / 2;
        const int part = rem % 2;
        if (pg[h] >= 0) {
          const uint16_t* src =
              a.vc + ((static_cast<int64_t>(pg[h]) * a.Hkv + kvh) * D + d) *
                         kPage + part * 8;
          u16x8_t v = *reinterpret_cast<const u16x8_t*>(src);
          // zero keys at or past k1 (they may hold anything)
          const int kbase = p0 + h * kPage + part * 8;
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (kbase + e >= k1) v[e] = 0;
          rv[u] = v;
        }
      }
    }
    return ok;
  }

  // Window tile: window rows j0 .. j0+31 (valid below W).
  __device__ void load_window(const AttnArgs& a, int b, int kvh, int j0) {
    const u16x8_t zero = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int u = 0; u < kPerThreadK; ++u) {
      const int ch = threadIdx.x + u * NT;
      rk[u] = zero;
      if (ch < kChunksK) {
        const int key = ch / (D / 8);
        const int col = ch % (D / 8);
        if (j0 + key < a.W) {
          const uint16_t* src =
              a.kw + ((static_cast<int64_t>(b) * a.W + j0 + key) * a.Hkv +
                      kvh) * D + col * 8;
          rk[u] = *reinterpret_cast<const u16x8_t*>(src);
        }
      }
    }
    // V rows are read token-major here and transposed on the LDS store
#pragma unroll
    for (int u = 0; u < kPerThreadV; ++u) {
      const int ch = threadIdx.x + u * NT;
      rv[u] = zero;
      if (ch < kChunksV) {
        const int key = ch / (D / 8);
        const int col = ch % (D / 8);
        if (j0 + key < a.W) {
          const uint16_t* src =
              a.vw + ((static_cast<int64_t>(b) * a.W + j0 + key) * a.Hkv +
                      kvh) * D + col * 8;
          rv[u] = *reinterpret_cast<const u16x8_t*>(src);
        }
      }
    }
  }

  __device__ void store_prefix(uint16_t* kl, uint16_t* vl) const {
#pragma unroll
    for (int u = 0; u < kPerThreadK; ++u) {
      const int ch = threadIdx.x + u * NT;
      if (ch < kChunksK) {
        const int key = ch / (D / 8);
        const int col = ch % (D / 8);
        *reinterpret_cast<u16x8_t*>(kl + key * Lds<D>::kPitch + col * 8) =
            rk[u];
      }
    }
#pragma unroll
    for (int u = 0; u < kPerThreadV; ++u) {
      const int ch = threadIdx.x + u * NT;
      if (ch < kChunksV) {
        const int h = ch / (2 * D);
        const int rem = ch % (2 * D);
        const int d = rem / 2;
        const int part = rem % 2;
        uint16_t* dst = vl + d * Lds<D>::vPitch + h * kPage + part * 8;
        const u16x4_t lo = {rv[u][0], rv[u][1], rv[u][2], rv[u][3]};
        const u16x4_t hi = {rv[u][4], rv[u][5], rv[u][6], rv[u][7]};
        *reinterpret_cast<u16x4_t*>(dst) = lo;
        *reinterpret_cast<u16x4_t*>(dst + 4) = hi;
      }
    }
  }

  __device__ void store_window(uint16_t* kl, uint16_t* vl) const {
#pragma unroll
    for (int u = 0; u < kPerThreadK; ++u) {
      const int ch = threadIdx.x + u * NT;
      if (ch < kChunksK) {
        const int key = ch / (D / 8);
        const int col = ch % (D / 8);
        *reinterpret_cast<u16x8_t*>(kl + key * Lds<D>::kPitch + col * 8) =
            rk[u];
      }
    }
#pragma unroll
    for (int u = 0; u < kPerThreadV; ++u) {
      const int ch = threadIdx.x + u * NT;
      if (ch < kChunksV) {
        const int key = ch / (D / 8);
        const int col = ch % (D / 8);
#pragma unroll
        for (int e = 0; e < 8; ++e)
          vl[(col * 8 + e) * Lds<D>::vPitch + key] = rv[u][e];
      }
    }
  }
};

template <int D, int NW>
__global__ __launch_bounds__(NW * kWave) void window_attn_kernel(AttnArgs a) {
  constexpr int NK = D / 16;   // k-steps of the score MFMA
  constexpr int NM = D / 32;   // 32-row blocks of O^T
  __shared__ __attribute__((aligned(16))) uint16_t s_k[2][Lds<D>::kElems];
  __shared__ __attribute__((aligned(16))) uint16_t s_v[2][Lds<D>::vElems];

  int wg = blockIdx.x;
  const int split = wg % a.nsplit;
  wg /= a.nsplit;
  const int qb = wg % a.qblocks;
  wg /= a.qblocks;
  const int kvh = wg % a.Hkv;
  const int b = wg / a.Hkv;

  int c;
  if (!seq_ok(a, b, c)) {
    if (a.status && threadIdx.x == 0 && split == 0 && qb == 0 && kvh == 0)
      atomicOr(a.status + b, WEDLM_SEQ_BAD_LEN);
    return;
  }
  const int nsplit_b = c > 0 ? (c + a.split_len - 1) / a.split_len : 1;
  if (split >= nsplit_b) return;
  const int k0 = split * a.split_len;
  const int k1 = min(c, k0 + a.split_len);
  const bool last = split == nsplit_b - 1;
  const int n_pre = k1 > k0 ? (k1 - k0 + kTileKeys - 1) / kTileKeys : 0;
  const int n_win = last ? (a.W + kTileKeys - 1) / kTileKeys : 0;
  const int n_tiles = n_pre + n_win;

  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int col = lane & 31;        // query column of this lane
  const int hf = lane >> 5;         // which half of the k slots
  const int rows = a.W * a.G;
  const int r = qb * (NW * 32) + wave * 32 + col;
  const bool rvalid = r < rows;
  const int qi = rvalid ? r / a.G : 0;          // physical window row
  const int qh = kvh * a.G + (rvalid ? r % a.G : 0);

  // queries as the B operand of S^T = K . Q^T
  bf16x8_t qf[NK];
  {
    const uint16_t* qp =
        a.q + ((static_cast<int64_t>(b) * a.W + qi) * a.Hq + qh) * D;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      u16x8_t v = {0, 0, 0, 0, 0, 0, 0, 0};
      if (rvalid) v = *reinterpret_cast<const u16x8_t*>(qp + kk * 16 + hf * 8);
      qf[kk] = __builtin_bit_cast(bf16x8_t, v);
    }
  }

  floatx16_t o[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[m][e] = 0.f;
  float m_run = kNegInf, l_run = 0.f;
  bool pages_ok = true;

  TileLoader<D, NW> ld;
  auto load_tile = [&](int t) {
    if (t < n_pre) pages_ok &= ld.load_prefix(a, b, kvh, k0 + t * kTileKeys, k1);
    else ld.load_window(a, b, kvh, (t - n_pre) * kTileKeys);
  };
  auto store_tile = [&](int t, int buf) {
    if (t < n_pre) ld.store_prefix(s_k[buf], s_v[buf]);
    else ld.store_window(s_k[buf], s_v[buf]);
  };

  if (n_tiles > 0) {
    load_tile(0);
    store_tile(0, 0);
  }
  __syncthreads();

  for (int t = 0; t < n_tiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < n_tiles) load_tile(t + 1);

    // scores of 32 keys x 32 queries
    floatx16_t acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.f;
    const uint16_t* kl = s_k[buf] + col * Lds<D>::kPitch + hf * 8;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      const bf16x8_t kf = __builtin_bit_cast(
          bf16x8_t, *reinterpret_cast<const u16x8_t*>(kl + kk * 16));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], acc, 0, 0, 0);
    }

    // mask, scale to log2 domain, online softmax
    const bool is_win = t >= n_pre;
    const int base = is_win ? (t - n_pre) * kTileKeys : k0 + t * kTileKeys;
    float mx = kNegInf;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int key = base + (e >> 2) * 8 + hf * 4 + (e & 3);
      const bool ok = is_win ? (key < a.W && key <= qi) : (key < k1);
      const float s = ok ? acc[e] * a.scale_log2 : kNegInf;
      acc[e] = s;
      mx = fmaxf(mx, s);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == kNegInf) ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float p = __builtin_amdgcn_exp2f(acc[e] - m_use);
      acc[e] = p;
      psum += p;
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[m][e] *= alpha;

    // O^T += V^T . P^T, two 16-key halves of the tile
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      bf16x8_t pf;
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[e] = static_cast<__bf16>(acc[h2 * 8 + e]);
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        const uint16_t* vl =
            s_v[buf] + (m * 32 + col) * Lds<D>::vPitch + h2 * 16 + hf * 4;
        const u16x4_t lo = *reinterpret_cast<const u16x4_t*>(vl);
        const u16x4_t hi = *reinterpret_cast<const u16x4_t*>(vl + 8);
        const u16x8_t vv = {lo[0], lo[1], lo[2], lo[3],
                            hi[0], hi[1], hi[2], hi[3]};
        o[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, vv), pf, o[m], 0, 0, 0);
      }
    }

    if (t + 1 < n_tiles) store_tile(t + 1, buf ^ 1);
    __syncthreads();
  }

  if (!pages_ok && a.status && threadIdx.x == 0)
    atomicOr(a.status + b, WEDLM_SEQ_BAD_PAGE);

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!rvalid) return;
  const int64_t rows_base =
      (static_cast<int64_t>(b) * a.Hkv + kvh) * a.rows_pad + r;
  if (a.nsplit == 1) {
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    uint16_t* op = a.out + ((static_cast<int64_t>(b) * a.W + qi) * a.Hq + qh) * D;
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int d = m * 32 + g4 * 8 + hf * 4;
        const u16x4_t v = {f32_to_bf16(o[m][g4 * 4 + 0] * inv),
                           f32_to_bf16(o[m][g4 * 4 + 1] * inv),
                           f32_to_bf16(o[m][g4 * 4 + 2] * inv),
                           f32_to_bf16(o[m][g4 * 4 + 3] * inv)};
        *reinterpret_cast<u16x4_t*>(op + d) = v;
      }
    if (a.lse && hf == 0)
      a.lse[(static_cast<int64_t>(b) * a.W + qi) * a.Hq + qh] =
          (m_run + __log2f(l_tot)) * kLn2;
  } else {
    float* wp = a.ws_o + (rows_base * a.nsplit + split) * D;
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int d = m * 32 + g4 * 8 + hf * 4;
        const floatx4_t v = {o[m][g4 * 4 + 0], o[m][g4 * 4 + 1],
                             o[m][g4 * 4 + 2], o[m][g4 * 4 + 3]};
        *reinterpret_cast<floatx4_t*>(wp + d) = v;
      }
    if (hf == 0) a.ws_ml[rows_base * a.nsplit + split] = make_float2(m_run, l_tot);
  }
}

// Merge of the split partials: one workgroup per (b, kv head, row), one
// thread per d.
template <int D>
__global__ __launch_bounds__(D) void attn_combine_kernel(AttnArgs a) {
  int wg = blockIdx.x;
  const int rows = a.W * a.G;
  const int r = wg % rows;
  wg /= rows;
  const int kvh = wg % a.Hkv;
  const int b = wg / a.Hkv;
  int c;
  if (!seq_ok(a, b, c)) return;
  const int nsplit_b = c > 0 ? (c + a.split_len - 1) / a.split_len : 1;
  const int64_t rows_base =
      (static_cast<int64_t>(b) * a.Hkv + kvh) * a.rows_pad + r;
  const float2* ml = a.ws_ml + rows_base * a.nsplit;
  float M = kNegInf;
  for (int s = 0; s < nsplit_b; ++s) M = fmaxf(M, ml[s].x);
  const float Mu = (M == kNegInf) ? 0.f : M;
  float L = 0.f, acc = 0.f;
  const int d = threadIdx.x;
  const float* op = a.ws_o + rows_base * a.nsplit * D + d;
  for (int s = 0; s < nsplit_b; ++s) {
    const float w = __builtin_amdgcn_exp2f(ml[s].x - Mu);
    L += w * ml[s].y;
    acc += w * op[static_cast<int64_t>(s) * D];
  }
  const int qi = r / a.G;
  const int qh = kvh * a.G + r % a.G;
  const float inv = L > 0.f ? 1.f / L : 0.f;
  a.out[((static_cast<int64_t>(b) * a.W + qi) * a.Hq + qh) * D + d] =
      f32_to_bf16(acc * inv);
  if (a.lse && d == 0)
    a.lse[(static_cast<int64_t>(b) * a.W + qi) * a.Hq + qh] =
        (M + __log2f(L)) * kLn2;
}

template <int D>
int launch(const AttnArgs& a, const Plan& p, hipStream_t st) {
  const int grid = a.nsplit * a.B * a.Hkv * a.qblocks;
  switch (p.nw) {
    case 8:
      hipLaunchKernelGGL((window_attn_kernel<D, 8>), dim3(grid), dim3(8 * kWave), 0, st, a);
      break;
    case 4:
      hipLaunchKernelGGL((window_attn_kernel<D, 4>), dim3(grid), dim3(4 * kWave), 0, st, a);
      break;
    case 2:
      hipLaunchKernelGGL((window_attn_kernel<D, 2>), dim3(grid), dim3(2 * kWave), 0, st, a);
      break;
    default:
      hipLaunchKernelGGL((window_attn_kernel<D, 1>), dim3(grid), dim3(kWave), 0, st, a);
      break;
  }
  WEDLM_LAUNCH_CHECK();
  if (a.nsplit > 1) {
    hipLaunchKernelGGL((attn_combine_kernel<D>), dim3(a.B * a.Hkv * a.W * a.G),
                       dim3(D), 0, st, a);
    WEDLM_LAUNCH_CHECK();
  }
  return WEDLM_OK;
}

bool shape_ok(int B, int W, int Hq, int Hkv, int D, int max_prefix) {
  return B >= 1 && W >= 1 && W <= WEDLM_MAX_WINDOW && Hkv >= 1 && Hq >= Hkv &&
         Hq % Hkv == 0 && (D == 64 || D == 128) && max_prefix >= 0 &&
         static_cast<int64_t>(B) * Hkv * W * (Hq / Hkv) < (1ll << 31);
}

}  // namespace

extern "C" size_t wedlm_window_attn_workspace_size(int32_t B, int32_t W,
                                                   int32_t Hq, int32_t Hkv,
                                                   int32_t D,
                                                   int32_t max_prefix_len) {
  if (!shape_ok(B, W, Hq, Hkv, D, max_prefix_len)) return 0;
  return make_plan(B, W, Hq, Hkv, D, max_prefix_len).ws_bytes;
}

extern "C" int wedlm_window_attn(
    const uint16_t* q_phys, const uint16_t* k_phys, const uint16_t* v_phys,
    const uint16_t* k_cache, const uint16_t* v_cache, int64_t num_pages,
    const int32_t* block_table, int32_t max_pages, const int32_t* prefix_len,
    int32_t B, int32_t W, int32_t Hq, int32_t Hkv, int32_t D,
    int32_t max_prefix_len, float softmax_scale, uint16_t* out, float* lse,
    int32_t* status, void* workspace, size_t workspace_bytes, void* stream) {
  if (!q_phys || !k_phys || !v_phys || !block_table || !prefix_len || !out)
    return WEDLM_E_ARG;
  if (!shape_ok(B, W, Hq, Hkv, D, max_prefix_len)) return WEDLM_E_SHAPE;
  if (max_prefix_len > 0 && (!k_cache || !v_cache || num_pages < 1 ||
                             max_pages < 1))
    return WEDLM_E_ARG;
  if (!(softmax_scale > 0.f) || !(softmax_scale < 1e30f)) return WEDLM_E_ARG;
  const Plan p = make_plan(B, W, Hq, Hkv, D, max_prefix_len);
  if (workspace_bytes < p.ws_bytes || (p.ws_bytes && !workspace))
    return WEDLM_E_WORKSPACE;
  AttnArgs a{};
  a.q = q_phys; a.kw = k_phys; a.vw = v_phys; a.kc = k_cache; a.vc = v_cache;
  a.bt = block_table; a.plen = prefix_len; a.out = out; a.lse = lse;
  a.status = status;
  a.num_pages = num_pages;
  a.B = B; a.W = W; a.Hq = Hq; a.Hkv = Hkv; a.G = Hq / Hkv;
  a.max_pages = max_pages; a.max_prefix = max_prefix_len;
  a.nsplit = p.nsplit; a.split_len = p.split_len; a.qblocks = p.qblocks;
  a.rows_pad = p.rows_pad;
  a.scale_log2 = softmax_scale * 1.4426950408889634f;
  if (p.nsplit > 1) {
    const size_t n = static_cast<size_t>(B) * Hkv * p.rows_pad * p.nsplit;
    char* base = static_cast<char*>(workspace);
    a.ws_o = reinterpret_cast<float*>(base);
    size_t off = (n * D * sizeof(float) + 255) & ~static_cast<size_t>(255);
    a.ws_ml = reinterpret_cast<float2*>(base + off);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  return D == 128 ? launch<128>(a, p, st) : launch<64>(a, p, st);
}
