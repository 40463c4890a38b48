// Causal GQA attention of the reordered window over the paged prefix cache
// (Sec. 4.1 "Context Awareness under Causal Masking"; Algorithm 1 Forward).
//
// Because the reordering has already moved every filled slot in front of
// every mask, the kernel is a plain causal prefill with a cache offset:
// physical row i sees all c prefix positions and window rows 0..i.  Logical
// positions entered only through RoPE (done by wedlm_reorder).
//
// Work decomposition (one GPU):
//   workgroup  = (sequence b, kv head, query block, prefix split)
//   query rows = the GQA-packed tile: row r = i*G + j is physical window
//                row i, query head kvh*G + j
//   each wave owns QB blocks of 32 query rows; all waves share 32-key tiles
//   of K and V staged in LDS.  S^T = K . Q^T and O^T += V^T . P^T run on
//   v_mfma_f32_32x32x16_bf16: keys are the M dimension of the score tile,
//   so a lane holds 16 scores of ONE query column and the row max / sum
//   need one cross-half exchange; each K or V operand read from LDS feeds
//   QB MFMAs.  The transposed V page layout makes V^T rows contiguous.
// Latency hiding: tiles go straight from HBM into an LDS ring of eight
//   tile slots (buffer loads with the LDS-destination bit, no register
//   staging), issued six tiles ahead; the workgroup synchronises once per
//   two tiles.
// Softmax: log2 domain, p = 2^(s*c - m) with c = softmax_scale * log2(e)
//   folded into one FMA per score.  There is no per-tile max: m, a column's
//   reference max, is the first tile's max and is raised only when the
//   running sum shows that some term exceeded 2^64 (never for scores that
//   grow by less than 64 log2 units past the first tile; a rare,
//   wave-uniform branch otherwise).
// Split-K: the prefix is split so that the grid fills the CUs; each split
//   writes its O normalised by its own sum, rounded to bf16 (the precision
//   of the P operand the MFMAs already take), with its running max and sum
//   in fp32, and a combine kernel merges them.  With a single split the
//   main kernel normalises and writes the output.
// Roofline: the KV stream, 4 * D * Hkv bytes per prefix position, read once
// per (sequence, kv head, query block); W*G query rows per kv head give an
// arithmetic intensity of W*G flop/byte (256 at W=64, G=4).
#include "common.h"
#include "internal.h"

#include <mutex>

using namespace wedlm;

namespace {

constexpr int kTileKeys = 32;       // keys per LDS tile (two 16-token pages)
// Page ids of one split's full tiles are staged in LDS, so the tile loop
// issues no scalar-cache loads (whose out-of-order return would make every
// wait on the LDS reads a full drain).  A split is at most this many pages.
constexpr int kMaxSplitPages = 2048;
constexpr float kLn2 = 0.69314718055994530942f;
// A prefix split holds at least this many 32-key tiles.
constexpr int kMinSplitTiles = 8;
// A column's running sum may reach this before its reference max is raised
// (every term 2^(s - m) is then at most 2^64, far inside fp32).
constexpr float kSumLimit = 18446744073709551616.0f;  // 2^64

struct AttnArgs {
  const uint16_t* q;      // [B, W, Hq, D]
  const uint16_t* kw;     // [B, W, Hkv, D]
  const uint16_t* vw;     // [B, W, Hkv, D]
  const uint16_t* kc;     // [P, Hkv, 16, D]
  const uint16_t* vc;     // [P, Hkv, D, 16]
  const int32_t* bt;      // [B, max_pages]
  const int32_t* plen;    // [B]
  uint16_t* out;          // [B, W, Hq, D], or packed tiles (packed != 0)
  float* lse;             // [B, W, Hq] or null
  int32_t* status;        // [B] or null
  uint16_t* ws_o;         // [B, Hkv, rows_pad, nsplit, D] bf16, normalised
  float2* ws_ml;          // [B, Hkv, rows_pad, nsplit]
  int64_t num_pages;
  int B, W, Hq, Hkv, G, max_pages, max_prefix, nsplit, qblocks,
      rows_pad;
  int packed;             // out as the B*W x Hq*D matrix in packed MFMA tiles
  // Paired blocks (pair_half = P > 0, W = 2P): "sequence" b is block
  // b % pair_K of sequence b / pair_K of a [seq][2 streams][pair_K blocks]
  // [P rows] layout; window rows 0..P-1 are the block of stream 0, rows
  // P..2P-1 the block of stream 1, and a window key is visible only to the
  // rows of its own half (causally).
  int pair_half, pair_K;
  // Workgroups take the sequences from the last one down (callers whose
  // later sequences have the longer prefixes: the longest start first)
  int rev;
  float scale_log2;       // softmax_scale * log2(e)
};

// Kernel shape for a given number of query rows per kv head.
struct Shape {
  int nw, qb;             // waves per workgroup, 32-row blocks per wave
};

Shape pick_shape(int rows) {
  if (rows <= 32) return {1, 1};
  if (rows <= 64) return {2, 1};
  if (rows <= 128) return {4, 1};
  return {8, 1};
}

struct Plan {
  Shape sh;
  bool two;               // four-wave workgroups, two per CU
  int rows, rows_per_wg, qblocks, rows_pad, nsplit;
  size_t ws_bytes;
};

Plan make_plan(int B, int W, int Hq, int Hkv, int D, int max_prefix) {
  Plan p{};
  const int G = Hq / Hkv;
  p.rows = W * G;
  p.sh = pick_shape(p.rows);
  p.rows_per_wg = 32 * p.sh.nw * p.sh.qb;
  p.qblocks = (p.rows + p.rows_per_wg - 1) / p.rows_per_wg;
  p.rows_pad = p.qblocks * p.rows_per_wg;
  const int tiles = (max_prefix + kTileKeys - 1) / kTileKeys;
  const int base = B * Hkv * p.qblocks;
  const int max_split = tiles / kMinSplitTiles > 1 ? tiles / kMinSplitTiles : 1;
  // Four-wave workgroups run two per CU when the grid reaches 512 (every
  // SIMD then holds two waves): without splitting, or by splitting when
  // the prefix bound allows 32 tiles per split (shorter prefixes measured
  // faster one workgroup per CU).  Otherwise about 256 workgroups.
  p.two = false;
  int nsplit = 1;
  if (p.sh.nw == 4) {
    const int need = (512 + base - 1) / base;
    if (need == 1 || tiles >= 32 * need) {
      p.two = true;
      nsplit = need;
    }
  }
  if (!p.two) {
    nsplit = (256 + base - 1) / base;
    if (nsplit > max_split) nsplit = max_split;
  }
  if (nsplit < 1) nsplit = 1;
  const int min_split = (tiles + kMaxSplitPages / 2 - 1) / (kMaxSplitPages / 2);
  if (nsplit < min_split) nsplit = min_split;
  p.nsplit = nsplit;
  if (p.nsplit == 1) {
    p.ws_bytes = 0;
  } else {
    const size_t n = static_cast<size_t>(B) * Hkv * p.rows_pad * p.nsplit;
    p.ws_bytes = n * D * sizeof(uint16_t) + 256 + n * sizeof(float2);
  }
  return p;
}

// Split of one sequence's prefix of c positions over the launch's nsplit
// slots: as many splits as keep at least 8 tiles each (one for an empty
// prefix), each of the same whole number of tiles.  Derived on the device
// from the sequence's own c, so a max_prefix_len far above the prefixes in
// use does not leave splits empty.  At most 1024 tiles per split (2048
// staged page ids), since the plan takes nsplit >= max tiles / 1024.
struct SeqSplit {
  int n, len;             // splits in use, positions per split
};

__device__ __forceinline__ SeqSplit seq_split(int c, int nsplit) {
  const int tiles = (c + kTileKeys - 1) / kTileKeys;
  int n = tiles / kMinSplitTiles;
  n = n < 1 ? 1 : (n > nsplit ? nsplit : n);
  const int per = tiles > 0 ? (tiles + n - 1) / n : 1;
  SeqSplit r;
  r.len = per * kTileKeys;
  r.n = c > 0 ? (c + r.len - 1) / r.len : 1;
  return r;
}

// Physical row of window row qi of sequence b: b*W + qi, or with paired
// blocks the row of that block and stream.
__device__ __forceinline__ int64_t win_row(const AttnArgs& a, int b, int qi) {
  if (a.pair_half == 0) return static_cast<int64_t>(b) * a.W + qi;
  const int sq = b / a.pair_K, k = b - sq * a.pair_K;
  const int half = qi >= a.pair_half ? 1 : 0;
  return ((static_cast<int64_t>(sq) * 2 + half) * a.pair_K + k) * a.pair_half +
         qi - half * a.pair_half;
}

// Sequence validity; bad lengths are reported and the sequence skipped.
__device__ __forceinline__ bool seq_ok(const AttnArgs& a, int b, int& c) {
  c = a.plen[b];
  return c >= 0 && c <= a.max_prefix &&
         static_cast<int64_t>(c) <= static_cast<int64_t>(a.max_pages) * kPage;
}

typedef __attribute__((address_space(1))) void gbl_void_t;
typedef __attribute__((address_space(4))) const int32_t const_i32_t;

// Values of x in this lane and in the lane 32 away (v_permlane32_swap).
__device__ __forceinline__ void xor32_pair(float x, float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x),
                                                  __float_as_uint(x), false,
                                                  false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}

// Wave-uniform read of a block-table entry through the scalar cache (the
// boundary tiles only; the tile loop reads page ids staged in LDS).
__device__ __forceinline__ int load_uniform(const int32_t* p, int idx) {
  idx = __builtin_amdgcn_readfirstlane(idx);
  return ((const_i32_t*)p)[idx];
}

// Layout of one 32-key tile in LDS (bytes).  The K halves of all slots
// form one region and the V^T halves another, each at most 64 KB, so every
// fragment read reaches any slot from one address register plus the
// instruction's 16-bit offset.
//   K   [32 keys][2D bytes]: 16-byte chunk c of key row r sits in slot
//       c ^ swz_k(r), so the 16 lanes of one ds_read_b128 pass (16 rows,
//       same chunk) hit 16 different slots.
//   V^T [2 pages][D rows][32 bytes]: chunk c (8 keys) of row d sits in slot
//       c ^ ((d >> 3) & 1); 16 lanes reading rows d..d+15 cover all banks.
template <int D>
struct Tile {
  static constexpr int kBytes = kTileKeys * D * 2;
  static constexpr int vBytes = kTileKeys * D * 2;
  static constexpr int bytes = kBytes + vBytes;
  static constexpr int nInstr = bytes / 1024;      // per tile, per workgroup
  static constexpr int kInstr = kBytes / 1024;
  static constexpr int keysPerInstr = 512 / D;     // K rows per instruction
  static constexpr int vInstrPerPage = D / 32;     // V^T rows: 32 per instr
  __device__ static __forceinline__ int swz_k(int r) {
    return D == 128 ? (r & 15) : ((r >> 1) & 7);
  }
  __device__ static __forceinline__ int k_off(int key, int c) {
    return key * 2 * D + ((c ^ swz_k(key)) << 4);
  }
  __device__ static __forceinline__ int v_off(int h, int d, int c) {
    return h * D * 32 + d * 32 + ((c ^ ((d >> 3) & 1)) << 4);
  }
};

// Key row of the score tile held in MFMA output row m: bits 2 and 3 of m
// swapped, so that output element e of a lane (hf = lane / 32) is key
// 16*(e/8) + 8*hf + e%8 and each lane's slice of P^T is 8 contiguous keys.
__device__ __forceinline__ int key_of_row(int m) {
  return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1);
}

// TWO: four-wave workgroups (128 query rows per kv head) that run two per
// CU, so that every SIMD holds two waves, on grids of at least 512
// workgroups: their ring is four slots (64 KB at D = 128), small enough for
// two workgroups' LDS, with a barrier after every tile.  Otherwise one
// workgroup per CU with an eight-slot ring, a barrier every two tiles and
// the K fragments read one step ahead.
template <int D, int NW, int QB, bool TWO>
__global__ __launch_bounds__(NW * kWave)
__attribute__((amdgpu_waves_per_eu(TWO ? 2 : 1)))
void window_attn_kernel(AttnArgs a) {
  using T = Tile<D>;
  constexpr int NK = D / 16;          // k-steps of the score MFMA
  constexpr int NM = D / 32;          // 32-row blocks of O^T
  static_assert(!TWO || NW == 4, "two per CU: four-wave workgroups");
  constexpr bool kTwo = TWO;
  constexpr bool kHoist = !kTwo;      // K fragments read one step ahead
  constexpr int kBarEvery = kTwo ? 1 : 2;   // iterations per barrier
  constexpr int NS = kTwo ? 4 : 8;    // LDS ring of 32-key tile slots
  constexpr int LEAD = kTwo ? 3 : NS - 2;   // tiles loaded ahead of the one scored
  static_assert(NS * T::kBytes <= 65536 && NS * T::vBytes <= 65536,
                "each LDS region within one 16-bit read offset");
  __shared__ __attribute__((aligned(1024))) char smem[NS * T::bytes];
  // K half and V^T half of LDS slot s
  auto kb = [&](int s) { return smem + s * T::kBytes; };
  auto vb = [&](int s) { return smem + NS * T::kBytes + s * T::vBytes; };
  __shared__ int32_t pg_lds[kMaxSplitPages];   // page ids of the full tiles

  int wg = blockIdx.x;
  const int split = wg % a.nsplit;
  wg /= a.nsplit;
  const int qb = wg % a.qblocks;
  wg /= a.qblocks;
  const int kvh = wg % a.Hkv;
  const int b = a.rev ? a.B - 1 - wg / a.Hkv : wg / a.Hkv;

  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int col = lane & 31;        // query column of this lane
  const int hf = lane >> 5;         // which half of the k slots
  const int rows = a.W * a.G;

  // ---- queries (B operand of S^T = K . Q^T), issued before the prefix
  // length is read: their addresses need only the workgroup's indices, so
  // their round trip overlaps those of the prefix length and page ids
  int qi[QB], qh[QB];
  bool rvalid[QB];
  bf16x8_t qf[QB][NK];
#pragma unroll
  for (int q = 0; q < QB; ++q) {
    const int r = qb * (NW * QB * 32) + (wave * QB + q) * 32 + col;
    rvalid[q] = r < rows;
    qi[q] = rvalid[q] ? r / a.G : 0;
    qh[q] = kvh * a.G + (rvalid[q] ? r % a.G : 0);
    const uint16_t* qp = a.q + (win_row(a, b, qi[q]) * a.Hq + qh[q]) * D;
    // padded rows (past W*G) read row 0's query; their outputs are dropped
#pragma unroll
    for (int kk = 0; kk < NK; ++kk)
      qf[q][kk] = __builtin_bit_cast(
          bf16x8_t, *reinterpret_cast<const u16x8_t*>(qp + kk * 16 + hf * 8));
  }

  int c;
  if (!seq_ok(a, b, c)) {
    if (a.status && threadIdx.x == 0 && split == 0 && qb == 0 && kvh == 0)
      atomicOr(a.status + b, WEDLM_SEQ_BAD_LEN);
    return;
  }
  const SeqSplit ss = seq_split(c, a.nsplit);
  const int nsplit_b = ss.n;
  if (split >= nsplit_b) return;
  const int k0 = split * ss.len;
  const int k1 = min(c, k0 + ss.len);
  const bool last = split == nsplit_b - 1;
  const int n_pre = k1 > k0 ? (k1 - k0 + kTileKeys - 1) / kTileKeys : 0;
  const int n_win = last ? (a.W + kTileKeys - 1) / kTileKeys : 0;


  // ---- tile loads.  A tile is four 4 KB blocks (D = 128; 2 KB for
  // D = 64): the K rows of page 0 and page 1, then the V^T rows of page 0
  // and page 1, each contiguous in the cache.  Chunk g = wave*64*CPT +
  // u*64 + lane (16 bytes) belongs to block g / BC, so the block of a
  // (wave, u) pair is wave-uniform: every load is a raw buffer load through
  // a per-page resource (scalar registers) at a fixed per-lane offset.
  // Full prefix tiles go straight to LDS: one load instruction fills 1 KB
  // of its slot in lane order, so the swizzle is applied on the HBM side
  // (lane l fetches the chunk whose swizzled home is byte 16*l of that
  // kilobyte).  The boundary tiles go through registers (g_voff: chunk
  // order in HBM, l_off: its swizzled LDS home).
  constexpr int NT = NW * kWave;
  constexpr int BC = kPage * D / 8;          // 16-byte chunks per block
  constexpr int CPT = 4 * BC / NT;           // chunks per thread per tile
  static_assert(4 * BC % NT == 0 && (64 * CPT) % 64 == 0, "chunk split");
  int g_voff[CPT], l_off[CPT], g_blk[CPT], d_voff[CPT];
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
#pragma unroll
  for (int u = 0; u < CPT; ++u) {
    const int g = wave * 64 * CPT + u * 64 + lane;
    const int blk = g / BC, c = g % BC;
    g_blk[u] = __builtin_amdgcn_readfirstlane(blk);
    g_voff[u] = c * 16;
    // c is also the 16-byte position within the block in LDS order
    if (blk < 2) {
      l_off[u] = T::k_off(blk * kPage + c / (D / 8), c % (D / 8));
      const int kip = c / (D / 8), slot = c % (D / 8);
      d_voff[u] = kip * 2 * D +
                  ((slot ^ T::swz_k(blk * kPage + kip)) << 4);
    } else {
      l_off[u] = T::v_off(blk - 2, c / 2, c % 2);
      const int d = c / 2, slot = c % 2;
      d_voff[u] = d * 32 + ((slot ^ ((d >> 3) & 1)) << 4);
    }
  }
  const int32_t* btb = a.bt + static_cast<int64_t>(b) * a.max_pages;
  bool pages_ok = true;
  constexpr int kBlockBytes = kPage * D * 2;
  const int np32 = a.num_pages > 0x7fffffff ? 0x7fffffff
                                            : static_cast<int>(a.num_pages);
  // page ids of full prefix tile t (staged in LDS, already checked)
  auto ids_of = [&](int t) {
    return *reinterpret_cast<const int2*>(pg_lds + 2 * t);
  };
  // a full prefix tile straight into LDS slot s: wave chunk g = wave*CPT +
  // u is kilobyte g of the slot's K half (g < 2 blocks) or of its V^T half
  // LDS byte address of smem: the loads' destinations are 32-bit LDS
  // offsets computed in scalar registers
  const uint32_t lds0 =
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_t*)smem));
  constexpr int kChunks = T::kBytes / 1024;
  auto dma_ids = [&](int2 ids, int s) {
    const int pg[2] = {__builtin_amdgcn_readfirstlane(ids.x),
                       __builtin_amdgcn_readfirstlane(ids.y)};
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
      const int blk = g_blk[u];
      const int h = blk & 1;
      const uint16_t* base = ((blk < 2) ? a.kc : a.vc) +
                             (static_cast<int64_t>(h ? pg[1] : pg[0]) * a.Hkv + kvh) *
                                 kPage * D;
      const int g = wave_u * CPT + u;
      const uint32_t dst =
          lds0 + ((blk < 2) ? s * T::kBytes + g * 1024
                            : NS * T::kBytes + s * T::vBytes +
                                  (g - kChunks) * 1024);
      load_to_lds16(buffer_rsrc(base, kBlockBytes), d_voff[u],
                    __builtin_amdgcn_readfirstlane(dst));
    }
  };
  auto stash = [&](const u16x8_t (&r)[CPT], int s) {
#pragma unroll
    for (int u = 0; u < CPT; ++u)
      *reinterpret_cast<u16x8_t*>((g_blk[u] < 2 ? kb(s) : vb(s)) + l_off[u]) =
          r[u];
  };

  floatx16_t o[QB][NM];
#pragma unroll
  for (int q = 0; q < QB; ++q)
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[q][m][e] = 0.f;
  // Per query column: m2 the reference max of s*c (log2 units; -inf before
  // any score), l_run the running sum of the weights.
  float m2[QB], l_run[QB];
#pragma unroll
  for (int q = 0; q < QB; ++q) {
    m2[q] = kNegInf;
    l_run[q] = 0.f;
  }
  const float c2 = a.scale_log2;

  // ---- the phases of one tile
  const int krow = key_of_row(col);
  // S^T for this wave's query columns from the K tile at stage sb, plain
  // (accumulator from zero)
  auto qk = [&](int slot, floatx16_t (&sc)[QB]) {
    const char* sb = kb(slot);
#pragma unroll
    for (int q = 0; q < QB; ++q)
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[q][e] = 0.f;
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      const bf16x8_t kf = __builtin_bit_cast(
          bf16x8_t, *reinterpret_cast<const u16x8_t*>(
                        sb + T::k_off(krow, 2 * kk + hf)));
#pragma unroll
      for (int q = 0; q < QB; ++q)
        sc[q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[q][kk], sc[q],
                                                        0, 0, 0);
    }
  };
  // Max over a column's 32 keys: 16 in this lane (a tree of v_max3), 16 in
  // the lane 32 away.
  auto col_max = [&](const floatx16_t& x) {
    float t[6];
#pragma unroll
    for (int g = 0; g < 5; ++g)
      t[g] = fmaxf(x[3 * g], fmaxf(x[3 * g + 1], x[3 * g + 2]));
    t[5] = x[15];
    float mx = fmaxf(t[0], fmaxf(t[1], t[2]));
    mx = fmaxf(mx, fmaxf(t[3], t[4]));
    mx = fmaxf(mx, t[5]);
    float x0, x1;
    xor32_pair(mx, x0, x1);
    return fmaxf(x0, x1);
  };
  // Scale the column's partial output and sum by alpha.
  auto rescale = [&](int q, float alpha) {
    l_run[q] *= alpha;
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[q][m][e] *= alpha;
  };
  // p = 2^(s*c - m2) for the 16 scores of this lane, P^T in bf16 (the B
  // operands of the two 16-key P.V MFMAs) and l_run + the sum of the 16
  // weights (a tree of fp32 adds).
  auto exp_tile = [&](const floatx16_t (&x)[QB], bf16x8_t (&pf)[QB][2],
                      float (&lsum)[QB]) {
#pragma unroll
    for (int q = 0; q < QB; ++q) {
      const float mc = m2[q] == kNegInf ? 0.f : m2[q];
      float pe[16];
#pragma unroll
      for (int e = 0; e < 16; ++e)
        pe[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(x[q][e], c2, -mc));
#pragma unroll
      for (int e = 0; e < 16; ++e)
        pf[q][e >> 3][e & 7] = static_cast<__bf16>(pe[e]);
      float ps[4];
#pragma unroll
      for (int g = 0; g < 4; ++g)
        ps[g] = (pe[4 * g] + pe[4 * g + 1]) + (pe[4 * g + 2] + pe[4 * g + 3]);
      lsum[q] = l_run[q] + ((ps[0] + ps[1]) + (ps[2] + ps[3]));
    }
  };
  // Boundary tiles: masked keys set to -inf, the reference max raised to
  // the tile's max where that is larger (rescaling the column), then the
  // weights as above.
  auto softmax_general = [&](floatx16_t (&sc)[QB], bool need_mask, int base,
                             int lim_pre, bool is_win, bf16x8_t (&pf)[QB][2]) {
#pragma unroll
    for (int q = 0; q < QB; ++q) {
      if (need_mask) {
        const int lim = is_win ? min(a.W - 1, qi[q]) : lim_pre;
        // paired blocks: a row of the second half sees no window key of
        // the first
        const int lo = is_win && a.pair_half > 0 && qi[q] >= a.pair_half
                           ? a.pair_half : 0;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = base + 16 * (e >> 3) + 8 * hf + (e & 7);
          sc[q][e] = key <= lim && key >= lo ? sc[q][e] : kNegInf;
        }
      }
      const float mx = col_max(sc[q]) * c2;
      if (ballot(mx > m2[q])) {
        const float m_new = fmaxf(m2[q], mx);
        rescale(q, m2[q] == kNegInf ? 0.f
                                    : __builtin_amdgcn_exp2f(m2[q] - m_new));
        m2[q] = m_new;
      }
    }
    float ls[QB];
    exp_tile(sc, pf, ls);
#pragma unroll
    for (int q = 0; q < QB; ++q) l_run[q] = ls[q];
  };
  // Full tiles whose running sum passed kSumLimit (some 2^(s*c - m) is
  // large): raise each column's reference max by the excess of its tile
  // max over it, rescale, and take the weights again.
  auto raise_max = [&](const floatx16_t (&sc)[QB], bf16x8_t (&pf)[QB][2],
                       float (&lsum)[QB]) {
#pragma unroll
    for (int q = 0; q < QB; ++q) {
      const float d = fmaxf(col_max(sc[q]) * c2 - m2[q], 0.f);
      rescale(q, __builtin_amdgcn_exp2f(-d));
      m2[q] += d;
    }
    exp_tile(sc, pf, lsum);
  };
  // V^T fragments of a tile: the A operands of the P.V MFMAs.  Row
  // m*32 + col keeps the swizzle bit of row col, so every fragment is this
  // lane's offset plus a constant (folded into the read's offset field).
  const int v_lane = T::v_off(0, col, hf);
  auto vread = [&](int slot, bf16x8_t (&vf)[2][NM]) {
    const char* sb = vb(slot) + v_lane;
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int m = 0; m < NM; ++m)
        vf[h2][m] = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const u16x8_t*>(
                          sb + h2 * D * 32 + m * 32 * 32));
  };
  // O^T += V^T . P^T
  auto pv = [&](const bf16x8_t (&vf)[2][NM], const bf16x8_t (&pf)[QB][2]) {
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int q = 0; q < QB; ++q)
          o[q][m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[h2][m], pf[q][h2],
                                                            o[q][m], 0, 0, 0);
  };

  // ---- full prefix tiles.  Tile t lives in LDS slot t % NS and is loaded
  // LEAD iterations before the one that scores it.  Iteration t runs the
  // weights of tile t (VALU) under the score MFMAs of tile t+1, then the
  // P.V MFMAs of tile t, and issues the loads of tile t+LEAD.  The K
  // fragments run one step ahead: those of tile t+2 are read as soon as
  // the score MFMAs of tile t+1 have taken theirs, so the next iteration's
  // score MFMAs never wait on LDS; the V fragments of tile t are read at
  // the top of iteration t, a whole softmax ahead of the P.V MFMAs that use
  // them.  The workgroup synchronises after odd iterations
  // only, each wave first waiting for its own loads of every tile up to
  // t+4 (the tiles read before the next barrier).  A slot is reloaded only
  // after a barrier that follows the last read of its previous tile
  // (NS = LEAD + 2), and no slot being loaded is read in the same
  // iteration.
  const bool partial_last = n_pre > 0 && (k1 - k0) % kTileKeys != 0;
  const int n_full = n_pre - (partial_last ? 1 : 0);
  floatx16_t sbuf[2][QB];     // scores of tile t in sbuf[t & 1]
  // Loads are unconditional (indices past the last full tile re-read that
  // tile into a slot nobody reads), so every wave issues the same number
  // of loads per iteration and the waits before the barriers are static.
  const int last_full = n_full - 1;
  // page ids of the full tiles into LDS; an invalid id is clamped to page 0
  // (in bounds) and reported
  for (int i = threadIdx.x; i < 2 * n_full; i += NT) {
    int id = btb[k0 / kPage + i];
    if (!(id >= 0 && id < np32)) {
      if (a.status) atomicOr(a.status + b, WEDLM_SEQ_BAD_PAGE);
      id = 0;
    }
    pg_lds[i] = id;
  }
  __syncthreads();
  // take delivery of the queries here, once (they were issued at the top and
  // have long arrived): later uses then see plain register values and the
  // tile loop never waits on these loads again
#pragma unroll
  for (int q = 0; q < QB; ++q)
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) asm volatile("" : "+v"(qf[q][kk]));

  // Tiles published at a barrier: with the K fragments one step ahead and
  // a barrier every two iterations, every tile up to t+4; without them and
  // a barrier every iteration, every tile up to t+2.
  constexpr int kHorizon = kBarEvery + (kHoist ? 2 : 1);
  constexpr int kInFlight = CPT * (LEAD - kHorizon);   // younger loads
  static_assert(LEAD > kHorizon, "publish horizon");
  static_assert(NS >= LEAD + kBarEvery, "slot reuse");
  // K fragments of the next tile to score
  bf16x8_t kf[NK];
  auto kread = [&](int slot) {
    const char* sb = kb(slot);
#pragma unroll
    for (int kk = 0; kk < NK; ++kk)
      kf[kk] = __builtin_bit_cast(
          bf16x8_t,
          *reinterpret_cast<const u16x8_t*>(sb + T::k_off(krow, 2 * kk + hf)));
  };
  // ---- boundary tiles: the partial last prefix tile (keys past k1 or on a
  // bad page are zeroed and masked), then the window tiles of the last
  // split (V transposed into V^T on the store).  They are scored before the
  // full tiles, in the ring's last slot (never among the first LEAD loads),
  // with their loads issued right after the first LEAD tile loads: the two
  // round trips overlap, and the boundary work is off the end of the split
  // (where it used to wait for its own loads after the last full tile).
  constexpr int kMaxTail = 1 + (WEDLM_MAX_WINDOW + kTileKeys - 1) / kTileKeys;
  const int n_tail = (partial_last ? 1 : 0) + n_win;
  constexpr int kTailSlot = NS - 1;
  static_assert(kTailSlot >= LEAD, "the tail slot is not among the first loads");
  int tail_lim = 0;
  u16x8_t tr[kMaxTail][CPT];
  auto tail_load = [&](int tt, u16x8_t (&r)[CPT]) {
    const bool is_win = !(partial_last && tt == 0);
    if (!is_win) {
      const int base = k0 + n_full * kTileKeys;
      int pg[2];
      bool pv2[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int id =
            (base + h * kPage < k1) ? load_uniform(btb, base / kPage + h) : -1;
        pv2[h] = id >= 0 && id < a.num_pages;
        if (base + h * kPage < k1 && !pv2[h]) pages_ok = false;
        pg[h] = pv2[h] ? id : 0;
      }
      const int lim =
          !pv2[0] ? base - 1 : (!pv2[1] ? min(k1, base + kPage) - 1 : k1 - 1);
      tail_lim = lim;
#pragma unroll
      for (int u = 0; u < CPT; ++u) {
        const int blk = g_blk[u];
        const int h = blk & 1;
        const bool isv = blk >= 2;
        const int64_t pbase =
            (static_cast<int64_t>(pg[h]) * a.Hkv + kvh) * kPage * D;
        u16x8_t v = *reinterpret_cast<const u16x8_t*>(
            (isv ? a.vc : a.kc) + pbase + g_voff[u] / 2);
        // first key of this chunk: one key per K chunk, eight per V chunk
        const int c = g_voff[u] / 16;
        const int kf = isv ? h * kPage + (c % 2) * 8 : h * kPage + c / (D / 8);
        const u16x8_t z = {0, 0, 0, 0, 0, 0, 0, 0};
        if (!isv) {
          v = (base + kf <= lim) ? v : z;
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            v[e] = (base + kf + e <= lim) ? v[e] : static_cast<uint16_t>(0);
        }
        r[u] = v;
      }
    } else {
      const int base = (tt - (partial_last ? 1 : 0)) * kTileKeys;
#pragma unroll
      for (int u = 0; u < CPT; ++u) {
        const int ch = static_cast<int>(threadIdx.x) + u * NT;
        const bool isv = ch >= kTileKeys * (D / 8);
        const int c2 = isv ? ch - kTileKeys * (D / 8) : ch;
        const int key = c2 / (D / 8);
        const int cc = c2 % (D / 8);
        u16x8_t v = {0, 0, 0, 0, 0, 0, 0, 0};
        if (base + key < a.W)
          v = *reinterpret_cast<const u16x8_t*>(
              (isv ? a.vw : a.kw) +
              (win_row(a, b, base + key) * a.Hkv + kvh) * D + cc * 8);
        r[u] = v;
      }
    }
  };
  auto tail_store = [&](int tt, const u16x8_t (&r)[CPT]) {
    const bool is_win = !(partial_last && tt == 0);
    if (!is_win) {
      stash(r, kTailSlot);
    } else {
#pragma unroll
      for (int u = 0; u < CPT; ++u) {
        const int ch = static_cast<int>(threadIdx.x) + u * NT;
        const bool isv = ch >= kTileKeys * (D / 8);
        const int c2 = isv ? ch - kTileKeys * (D / 8) : ch;
        const int key = c2 / (D / 8);
        const int cc = c2 % (D / 8);
        if (!isv) {
          *reinterpret_cast<u16x8_t*>(kb(kTailSlot) + T::k_off(key, cc)) = r[u];
        } else {
          const int h = key / kPage, kk = key % kPage;
#pragma unroll
          for (int e = 0; e < 8; ++e)
            *reinterpret_cast<uint16_t*>(vb(kTailSlot) +
                                         T::v_off(h, cc * 8 + e, kk / 8) +
                                         (kk % 8) * 2) = r[u][e];
        }
      }
    }
  };
  auto tail_tiles = [&]() {
#pragma unroll
    for (int tt = 0; tt < kMaxTail; ++tt)
      if (tt < n_tail) tail_load(tt, tr[tt]);
#pragma unroll
    for (int tt = 0; tt < kMaxTail; ++tt) {
      if (tt < n_tail) {
        const bool is_win = !(partial_last && tt == 0);
        const int base = is_win ? (tt - (partial_last ? 1 : 0)) * kTileKeys
                                : k0 + n_full * kTileKeys;
        __syncthreads();   // every wave is done with the slot's last tile
        tail_store(tt, tr[tt]);
        __syncthreads();
        qk(kTailSlot, sbuf[0]);
        bf16x8_t pf[QB][2], vf[2][NM];
        softmax_general(sbuf[0], true, base, tail_lim, is_win, pf);
        vread(kTailSlot, vf);
        pv(vf, pf);
      }
    }
    __syncthreads();       // the slot is free for the ring's loads
  };
  if (n_full > 0) {
#pragma unroll
    for (int j = 0; j < LEAD; ++j)
      dma_ids(ids_of(min(j, last_full)), j);
  }
  if (n_tail > 0) tail_tiles();
  if (n_full > 0) {
    wait_vmcnt<kInFlight>();
    __syncthreads();
    qk(0, sbuf[0]);
    if constexpr (kHoist) kread(1);
    // the first full tile's max is each column's reference max, or raises
    // the one the boundary tiles set (the column rescaled)
#pragma unroll
    for (int q = 0; q < QB; ++q) {
      const float mx = col_max(sbuf[0][q]) * c2;
      if (mx > m2[q]) {
        rescale(q, m2[q] == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m2[q] - mx));
        m2[q] = mx;
      }
    }
  }
  // page ids of the next load, read one iteration ahead of their use
  int2 nid = ids_of(min(LEAD, max(last_full, 0)));
  // Iteration t (j = t mod U, a compile-time constant after unrolling, so
  // LDS slots and score buffers are static).  The body is one macro used
  // twice below; written as a lambda instead, the compiler allocates
  // registers differently and spills inside the main loop.
#define WEDLM_TILE_ITER                                                   \
    if constexpr (!kHoist) kread((j + 1) % NS);                           \
    bf16x8_t vf[2][NM];                                                   \
    vread(j % NS, vf);                                                    \
    {                                                                     \
      const int2 cur = nid;                                               \
      nid = ids_of(min(t + LEAD + 1, last_full));                         \
      dma_ids(cur, (j + LEAD) % NS);                                      \
    }                                                                     \
    /* one scheduling region: the score MFMAs of tile t+1 interleaved     */\
    /* with the weights of tile t                                        */\
    bf16x8_t pf[QB][2];                                                   \
    float lsum[QB];                                                       \
    _Pragma("unroll")                                                     \
    for (int q = 0; q < QB; ++q) {                                        \
      sbuf[(j + 1) & 1][q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(     \
          kf[0], qf[q][0], floatx16_t{}, 0, 0, 0);                        \
      _Pragma("unroll")                                                   \
      for (int kk = 1; kk < NK; ++kk)                                     \
        sbuf[(j + 1) & 1][q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(   \
            kf[kk], qf[q][kk], sbuf[(j + 1) & 1][q], 0, 0, 0);            \
    }                                                                     \
    exp_tile(sbuf[j & 1], pf, lsum);                                      \
    _Pragma("unroll")                                                     \
    for (int i = 0; i < NK * QB; ++i) {                                   \
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   /* one MFMA  */\
      __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);   /* two VALU  */\
    }                                                                     \
    {                                                                     \
      bool big = false;                                                   \
      _Pragma("unroll")                                                   \
      for (int q = 0; q < QB; ++q) big = big || (lsum[q] > kSumLimit);    \
      if (ballot(big)) raise_max(sbuf[j & 1], pf, lsum);                  \
    }                                                                     \
    _Pragma("unroll")                                                     \
    for (int q = 0; q < QB; ++q) l_run[q] = lsum[q];                      \
    /* K fragments of tile t+2 (a re-read tile past the last full one) */ \
    if constexpr (kHoist) kread((j + 2) % NS);                            \
    pv(vf, pf);                                                           \
    if ((j % kBarEvery) == kBarEvery - 1) {                               \
      __builtin_amdgcn_sched_barrier(0);                                  \
      wait_vmcnt<kInFlight>();                                            \
      __syncthreads();                                                    \
    }
  {
  constexpr int U = NS % kBarEvery == 0 ? NS : kBarEvery * NS;
  // whole groups of U tiles with no exit inside, so the loop carries the
  // same in-flight loads around its back edge as it receives on entry and
  // the compiler's waits stay partial; then the remaining tiles
  const int ngroups = n_full / U;
  for (int t0 = 0; t0 < ngroups * U; t0 += U) {
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int t = t0 + j;
      WEDLM_TILE_ITER
    }
  }
  {
    const int t0 = ngroups * U;
#pragma unroll
    for (int j = 0; j < U; ++j) {
      const int t = t0 + j;
      if (t >= n_full) goto tiles_done;
      WEDLM_TILE_ITER
    }
  }
  }
#undef WEDLM_TILE_ITER
tiles_done:
  wait_vmcnt<0>();   // surplus fetches retire before the output is written

  if (!pages_ok && a.status && threadIdx.x == 0)
    atomicOr(a.status + b, WEDLM_SEQ_BAD_PAGE);

#pragma unroll
  for (int q = 0; q < QB; ++q) {
    float l0, l1;
    xor32_pair(l_run[q], l0, l1);
    const float l_tot = l0 + l1;
    if (!rvalid[q]) continue;
    const int r = qb * (NW * QB * 32) + (wave * QB + q) * 32 + col;
    const int64_t rows_base =
        (static_cast<int64_t>(b) * a.Hkv + kvh) * a.rows_pad + r;
    if (a.nsplit == 1) {
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      const int64_t t = win_row(a, b, qi[q]);
      uint16_t* op = a.out + (t * a.Hq + qh[q]) * D;
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const int d = m * 32 + g4 * 8 + hf * 4;
          const u16x4_t v = {f32_to_bf16(o[q][m][g4 * 4 + 0] * inv),
                             f32_to_bf16(o[q][m][g4 * 4 + 1] * inv),
                             f32_to_bf16(o[q][m][g4 * 4 + 2] * inv),
                             f32_to_bf16(o[q][m][g4 * 4 + 3] * inv)};
          *reinterpret_cast<u16x4_t*>(
              a.packed ? a.out + packed_off(t, qh[q] * D + d, a.Hq * D)
                       : op + d) = v;
        }
      if (a.lse && hf == 0)
        a.lse[t * a.Hq + qh[q]] = (m2[q] + __log2f(l_tot)) * kLn2;
    } else {
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      uint16_t* wp = a.ws_o + (rows_base * a.nsplit + split) * D;
#pragma unroll
      for (int m = 0; m < NM; ++m)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const int d = m * 32 + g4 * 8 + hf * 4;
          const u16x4_t v = {f32_to_bf16(o[q][m][g4 * 4 + 0] * inv),
                             f32_to_bf16(o[q][m][g4 * 4 + 1] * inv),
                             f32_to_bf16(o[q][m][g4 * 4 + 2] * inv),
                             f32_to_bf16(o[q][m][g4 * 4 + 3] * inv)};
          *reinterpret_cast<u16x4_t*>(wp + d) = v;
        }
      if (hf == 0)
        a.ws_ml[rows_base * a.nsplit + split] =
            make_float2(m2[q], l_tot);   // log2 units
    }
  }
}

// Merge of the split partials: D/8 threads per (b, kv head, row) and slot
// group, each owning eight consecutive d (one 16-byte load per split); the
// SG slot groups of a row take the splits s = sg, sg + SG, ... and sit on
// neighbouring lanes of one wave.  O = sum_s 2^(m_s - M) l_s O_s /
// sum_s 2^(m_s - M) l_s over the splits s of the row (O_s normalised by
// l_s).  Every thread loads its (m, l) pairs and up to eight partial
// vectors before any is used, so one memory round trip covers up to 8 SG
// splits; the max and the sums are then combined across the slot groups
// with lane exchanges, in a fixed order.
constexpr int kCombineThreads = 256;

template <int D, int SG>
__global__ __launch_bounds__(kCombineThreads) void attn_combine_kernel(AttnArgs a) {
  constexpr int TPR = D / 8;                       // d groups of a row
  constexpr int TPW = TPR * SG;                    // threads per row
  static_assert(TPW <= kWave && kWave % TPW == 0, "a row within one wave");
  constexpr int RPW = kCombineThreads / TPW;       // rows per workgroup
  constexpr int kFast = 8;                         // slots per thread at once
  const int rows = a.W * a.G;
  const int64_t gr = static_cast<int64_t>(blockIdx.x) * RPW + threadIdx.x / TPW;
  // whole rows (aligned groups of TPW lanes) leave together, so the lane
  // exchanges below only ever read lanes of the same row
  if (gr >= static_cast<int64_t>(a.B) * a.Hkv * rows) return;
  const int r = static_cast<int>(gr % rows);
  const int bk = static_cast<int>(gr / rows);
  const int kvh = bk % a.Hkv;
  const int b = bk / a.Hkv;
  const int sg = (threadIdx.x % TPW) / TPR;
  const int d = (threadIdx.x % TPR) * 8;
  const int64_t rows_base =
      (static_cast<int64_t>(b) * a.Hkv + kvh) * a.rows_pad + r;
  const float2* ml = a.ws_ml + rows_base * a.nsplit;
  const uint16_t* op = a.ws_o + rows_base * a.nsplit * D + d;
  // the first slots are loaded before the prefix length is known (slots
  // past this sequence's splits are in the workspace and their values are
  // never used), so both round trips overlap
  float2 mls[kFast];
  u16x8_t vs[kFast];
#pragma unroll
  for (int i = 0; i < kFast; ++i) {
    const int s = sg + SG * i;
    if (s < a.nsplit) {
      mls[i] = ml[s];
      vs[i] = *reinterpret_cast<const u16x8_t*>(op + static_cast<int64_t>(s) * D);
    }
  }
  int c;
  if (!seq_ok(a, b, c)) return;                    // uniform over the row
  const int nsplit_b = seq_split(c, a.nsplit).n;
  float M = kNegInf;
#pragma unroll
  for (int i = 0; i < kFast; ++i)
    if (sg + SG * i < nsplit_b) M = fmaxf(M, mls[i].x);
  for (int s = sg + SG * kFast; s < nsplit_b; s += SG) M = fmaxf(M, ml[s].x);
#pragma unroll
  for (int off = TPR; off < TPW; off <<= 1) M = fmaxf(M, __shfl_xor(M, off));
  const float Mu = (M == kNegInf) ? 0.f : M;
  float L = 0.f;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < kFast; ++i) {
    if (sg + SG * i < nsplit_b) {
      const float w = __builtin_amdgcn_exp2f(mls[i].x - Mu) * mls[i].y;
      L += w;
#pragma unroll
      for (int k = 0; k < 8; ++k) acc[k] += w * bf16_to_f32(vs[i][k]);
    }
  }
  for (int s = sg + SG * kFast; s < nsplit_b; s += SG) {
    const float w = __builtin_amdgcn_exp2f(ml[s].x - Mu) * ml[s].y;
    L += w;
    const u16x8_t v = *reinterpret_cast<const u16x8_t*>(op + static_cast<int64_t>(s) * D);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] += w * bf16_to_f32(v[k]);
  }
#pragma unroll
  for (int off = TPR; off < TPW; off <<= 1) {
    L += __shfl_xor(L, off);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] += __shfl_xor(acc[k], off);
  }
  if (sg != 0) return;
  const int qi = r / a.G;
  const int qh = kvh * a.G + r % a.G;
  const int64_t t = win_row(a, b, qi);
  const int64_t orow = t * a.Hq + qh;
  const float inv = L > 0.f ? 1.f / L : 0.f;
  u16x8_t o8;
#pragma unroll
  for (int k = 0; k < 8; ++k) o8[k] = f32_to_bf16(acc[k] * inv);
  *reinterpret_cast<u16x8_t*>(
      a.packed ? a.out + packed_off(t, qh * D + d, a.Hq * D)
               : a.out + orow * D + d) = o8;
  if (a.lse && d == 0) a.lse[orow] = (M + __log2f(L)) * kLn2;
}

// Slot groups of the combine: enough that each thread loads at most eight
// splits at once, at most one wave per row.
template <int D, int SG>
void launch_combine(const AttnArgs& a, hipStream_t st) {
  const int64_t total_rows = static_cast<int64_t>(a.B) * a.Hkv * a.W * a.G;
  constexpr int rpw = kCombineThreads / (D / 8 * SG);
  hipLaunchKernelGGL((attn_combine_kernel<D, SG>),
                     dim3(static_cast<unsigned>((total_rows + rpw - 1) / rpw)),
                     dim3(kCombineThreads), 0, st, a);
}

template <int D>
void combine(const AttnArgs& a, hipStream_t st) {
  constexpr int kMaxSG = kWave / (D / 8);
  const int sg = a.nsplit <= 8 ? 1 : a.nsplit <= 16 ? 2 : a.nsplit <= 32 ? 4 : 8;
  switch (sg < kMaxSG ? sg : kMaxSG) {
    case 1: launch_combine<D, 1>(a, st); break;
    case 2: launch_combine<D, 2>(a, st); break;
    case 4: launch_combine<D, 4>(a, st); break;
    default: launch_combine<D, kMaxSG>(a, st); break;
  }
}

template <int D>
int launch(const AttnArgs& a, const Plan& p, hipStream_t st) {
  const int grid = a.nsplit * a.B * a.Hkv * a.qblocks;
  switch (p.sh.nw) {
    case 8:
      hipLaunchKernelGGL((window_attn_kernel<D, 8, 1, false>), dim3(grid),
                         dim3(8 * kWave), 0, st, a);
      break;
    case 4:
      if (p.two)
        hipLaunchKernelGGL((window_attn_kernel<D, 4, 1, true>), dim3(grid),
                           dim3(4 * kWave), 0, st, a);
      else
        hipLaunchKernelGGL((window_attn_kernel<D, 4, 1, false>), dim3(grid),
                           dim3(4 * kWave), 0, st, a);
      break;
    case 2:
      hipLaunchKernelGGL((window_attn_kernel<D, 2, 1, false>), dim3(grid),
                         dim3(2 * kWave), 0, st, a);
      break;
    default:
      hipLaunchKernelGGL((window_attn_kernel<D, 1, 1, false>), dim3(grid),
                         dim3(kWave), 0, st, a);
      break;
  }
  WEDLM_LAUNCH_CHECK();
  if (a.nsplit > 1) {
    combine<D>(a, st);
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

// Split-K partials of wedlm_window_attn_noalloc: one array per device (each
// GPU the library runs on holds its own copy until the process ends).  In
// host code the name is only a handle, never a device address: the address
// comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) char scratch[WEDLM_ATTN_SCRATCH_BYTES];

namespace {

constexpr size_t kScratchBytes = WEDLM_ATTN_SCRATCH_BYTES;

// The entry point's work; `workspace` holds at least the plan's bytes
// (checked by the callers).
int window_attn_impl(
    const uint16_t* q_phys, const uint16_t* k_phys, const uint16_t* v_phys,
    const uint16_t* k_cache, const uint16_t* v_cache, int64_t num_pages,
    const int32_t* block_table, int32_t max_pages, const int32_t* prefix_len,
    int32_t B, int32_t W, int32_t Hq, int32_t Hkv, int32_t D,
    int32_t max_prefix_len, float softmax_scale, uint16_t* out, float* lse,
    int32_t* status, const Plan& p, void* workspace, hipStream_t st,
    bool packed = false, int pair_half = 0, int pair_K = 0, bool rev = false) {
  AttnArgs a{};
  a.packed = packed ? 1 : 0;
  a.pair_half = pair_half;
  a.pair_K = pair_K;
  a.rev = rev ? 1 : 0;
  a.q = q_phys; a.kw = k_phys; a.vw = v_phys; a.kc = k_cache; a.vc = v_cache;
  a.bt = block_table; a.plen = prefix_len; a.out = out; a.lse = lse;
  a.status = status;
  a.num_pages = num_pages;
  a.B = B; a.W = W; a.Hq = Hq; a.Hkv = Hkv; a.G = Hq / Hkv;
  a.max_pages = max_pages; a.max_prefix = max_prefix_len;
  a.nsplit = p.nsplit; a.qblocks = p.qblocks;
  a.rows_pad = p.rows_pad;
  a.scale_log2 = softmax_scale * 1.4426950408889634f;
  if (p.nsplit > 1) {
    const size_t n = static_cast<size_t>(B) * Hkv * p.rows_pad * p.nsplit;
    char* base = static_cast<char*>(workspace);
    a.ws_o = reinterpret_cast<uint16_t*>(base);
    size_t off = (n * D * sizeof(uint16_t) + 255) & ~static_cast<size_t>(255);
    a.ws_ml = reinterpret_cast<float2*>(base + off);
  }
  return D == 128 ? launch<128>(a, p, st) : launch<64>(a, p, st);
}

// Host-side checks shared by both entry points.
int check_args(const uint16_t* q_phys, const uint16_t* k_phys,
               const uint16_t* v_phys, const uint16_t* k_cache,
               const uint16_t* v_cache, int64_t num_pages,
               const int32_t* block_table, int32_t max_pages,
               const int32_t* prefix_len, int32_t B, int32_t W, int32_t Hq,
               int32_t Hkv, int32_t D, int32_t max_prefix_len,
               float softmax_scale, const uint16_t* out) {
  if (!q_phys || !k_phys || !v_phys || !block_table || !prefix_len || !out)
    return WEDLM_E_ARG;
  if (!shape_ok(B, W, Hq, Hkv, D, max_prefix_len)) return WEDLM_E_SHAPE;
  if (max_prefix_len > 0 && (!k_cache || !v_cache || num_pages < 1 ||
                             max_pages < 1))
    return WEDLM_E_ARG;
  if (!(softmax_scale > 0.f) || !(softmax_scale < 1e30f)) return WEDLM_E_ARG;
  return WEDLM_OK;
}

constexpr int kMaxDevices = 64;
void* g_scratch_ptr[kMaxDevices];
std::once_flag g_scratch_once[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

// Device address of this device's scratch array (nullptr on failure).
void* scratch_ptr(int dev) {
  std::call_once(g_scratch_once[dev], [dev] {
    void* ptr = nullptr;
    g_scratch_err[dev] =
        hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    g_scratch_ptr[dev] = g_scratch_err[dev] == hipSuccess ? ptr : nullptr;
  });
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" int wedlm_window_attn_noalloc(
    const uint16_t* q_phys, const uint16_t* k_phys, const uint16_t* v_phys,
    const uint16_t* k_cache, const uint16_t* v_cache, int64_t num_pages,
    const int32_t* block_table, int32_t max_pages, const int32_t* prefix_len,
    int32_t B, int32_t W, int32_t Hq, int32_t Hkv, int32_t D,
    int32_t max_prefix_len, float softmax_scale, uint16_t* out, float* lse,
    int32_t* status, void* stream) {
  const int e = check_args(q_phys, k_phys, v_phys, k_cache, v_cache,
                           num_pages, block_table, max_pages, prefix_len, B,
                           W, Hq, Hkv, D, max_prefix_len, softmax_scale, out);
  if (e != WEDLM_OK) return e;
  const Plan p = make_plan(B, W, Hq, Hkv, D, max_prefix_len);
  if (p.ws_bytes > kScratchBytes) return WEDLM_E_SCRATCH;
  void* ws = nullptr;
  if (p.ws_bytes) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
      return WEDLM_E_DEVICE;
    ws = scratch_ptr(dev);
    if (!ws) return WEDLM_E_DEVICE;
  }
  return window_attn_impl(q_phys, k_phys, v_phys, k_cache, v_cache,
                          num_pages, block_table, max_pages, prefix_len, B, W,
                          Hq, Hkv, D, max_prefix_len, softmax_scale, out, lse,
                          status, p, ws, static_cast<hipStream_t>(stream));
}

extern "C" int wedlm_window_attn(
    const uint16_t* q_phys, const uint16_t* k_phys, const uint16_t* v_phys,
    const uint16_t* k_cache, const uint16_t* v_cache, int64_t num_pages,
    const int32_t* block_table, int32_t max_pages, const int32_t* prefix_len,
    int32_t B, int32_t W, int32_t Hq, int32_t Hkv, int32_t D,
    int32_t max_prefix_len, float softmax_scale, uint16_t* out, float* lse,
    int32_t* status, void* workspace, size_t workspace_bytes, void* stream) {
  const int e = check_args(q_phys, k_phys, v_phys, k_cache, v_cache,
                           num_pages, block_table, max_pages, prefix_len, B,
                           W, Hq, Hkv, D, max_prefix_len, softmax_scale, out);
  if (e != WEDLM_OK) return e;
  const Plan p = make_plan(B, W, Hq, Hkv, D, max_prefix_len);
  if (workspace_bytes < p.ws_bytes || (p.ws_bytes && !workspace))
    return WEDLM_E_WORKSPACE;
  return window_attn_impl(q_phys, k_phys, v_phys, k_cache, v_cache,
                          num_pages, block_table, max_pages, prefix_len, B, W,
                          Hq, Hkv, D, max_prefix_len, softmax_scale, out, lse,
                          status, p, workspace,
                          static_cast<hipStream_t>(stream));
}

// wedlm_window_attn with the output in the packed MFMA tile layout of the
// projections (the B*W x Hq*D matrix, ceil(B*W/32) row tiles; rows past B*W
// are not written), for the decoder, whose output projection reads it so.
int wedlm::window_attn_packed(
    const uint16_t* q_phys, const uint16_t* k_phys, const uint16_t* v_phys,
    const uint16_t* k_cache, const uint16_t* v_cache, int64_t num_pages,
    const int32_t* block_table, int32_t max_pages, const int32_t* prefix_len,
    int32_t B, int32_t W, int32_t Hq, int32_t Hkv, int32_t D,
    int32_t max_prefix_len, float softmax_scale, uint16_t* out_packed,
    int32_t* status, void* workspace, size_t workspace_bytes, void* stream) {
  const int e = check_args(q_phys, k_phys, v_phys, k_cache, v_cache,
                           num_pages, block_table, max_pages, prefix_len, B,
                           W, Hq, Hkv, D, max_prefix_len, softmax_scale,
                           out_packed);
  if (e != WEDLM_OK) return e;
  if ((static_cast<int64_t>(Hq) * D) % 64 != 0) return WEDLM_E_SHAPE;
  const Plan p = make_plan(B, W, Hq, Hkv, D, max_prefix_len);
  if (workspace_bytes < p.ws_bytes || (p.ws_bytes && !workspace))
    return WEDLM_E_WORKSPACE;
  return window_attn_impl(q_phys, k_phys, v_phys, k_cache, v_cache,
                          num_pages, block_table, max_pages, prefix_len, B, W,
                          Hq, Hkv, D, max_prefix_len, softmax_scale,
                          out_packed, nullptr, status, p, workspace,
                          static_cast<hipStream_t>(stream), true);
}

// The attention of paired blocks (Sec. 4.2's memory block k and prediction
// block k share the prefix of the k*P memory positions before them): one
// window of 2P rows per pair over that prefix, the two halves masked apart.
// The prefix grows with the block index, so the workgroups take the pairs
// from the last down: the longest run first and the short ones fill the
// end of the grid.
int wedlm::window_attn_pairs(
    const uint16_t* q, const uint16_t* k, const uint16_t* v,
    const uint16_t* k_cache, const uint16_t* v_cache, int64_t num_pages,
    const int32_t* block_table, int32_t max_pages, const int32_t* prefix_len,
    int32_t n_seq, int32_t blocks, int32_t P, int32_t Hq, int32_t Hkv,
    int32_t D, int32_t max_prefix_len, float softmax_scale, uint16_t* out,
    float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  if (n_seq < 1 || blocks < 1 || P < 1 || 2 * P > WEDLM_MAX_WINDOW)
    return WEDLM_E_SHAPE;
  const int64_t pairs = static_cast<int64_t>(n_seq) * blocks;
  if (pairs > (1 << 30)) return WEDLM_E_SHAPE;
  const int B = static_cast<int>(pairs), W = 2 * P;
  const int e = check_args(q, k, v, k_cache, v_cache, num_pages, block_table,
                           max_pages, prefix_len, B, W, Hq, Hkv, D,
                           max_prefix_len, softmax_scale, out);
  if (e != WEDLM_OK) return e;
  const Plan p = make_plan(B, W, Hq, Hkv, D, max_prefix_len);
  if (workspace_bytes < p.ws_bytes || (p.ws_bytes && !workspace))
    return WEDLM_E_WORKSPACE;
  return window_attn_impl(q, k, v, k_cache, v_cache, num_pages, block_table,
                          max_pages, prefix_len, B, W, Hq, Hkv, D,
                          max_prefix_len, softmax_scale, out, lse, nullptr, p,
                          workspace, static_cast<hipStream_t>(stream), false,
                          P, blocks, true);
}

size_t wedlm::window_attn_pairs_workspace_size(int32_t n_seq, int32_t blocks,
                                               int32_t P, int32_t Hq,
                                               int32_t Hkv, int32_t D,
                                               int32_t max_prefix_len) {
  if (n_seq < 1 || blocks < 1 || P < 1 || 2 * P > WEDLM_MAX_WINDOW) return 0;
  const int64_t pairs = static_cast<int64_t>(n_seq) * blocks;
  if (pairs > (1 << 30)) return 0;
  if (!shape_ok(static_cast<int>(pairs), 2 * P, Hq, Hkv, D, max_prefix_len))
    return 0;
  return make_plan(static_cast<int>(pairs), 2 * P, Hq, Hkv, D, max_prefix_len)
      .ws_bytes;
}
