// The decoder around the step: embedding, RMSNorm, the projections (a
// weight-streaming GEMM with fused epilogues), per-head RMSNorm + RoPE of
// the queries and keys, and the L-layer forward that strings them together
// with the window attention and the fused output layer.  WeDLM-8B keeps its
// Qwen3-8B backbone (Sec. 6.1); the forward runs the whole window in the
// physical order of Eq. (5)/(6), positions from Eq. (2).
//
// GEMM (gemm_kernel): out[t][n] = sum_k x[t][k] * w[n][k] for the window's
// M = B*W rows.  At decode sizes the weights are the HBM stream and every
// weight byte is used by all M rows, so a workgroup owns one 32-feature
// block (two for SwiGLU: the gate block and the matching up block) and one
// group of 32*NB rows, and its 8 waves split K: wave w walks its own run of
// 64-wide k steps with every load in registers PF steps ahead, no LDS and no
// barrier in the loop.  The 8 partial tiles are summed through LDS in a fixed
// order (deterministic) and the epilogue writes bf16, adds into the fp32
// residual stream, or applies silu(gate) * up.
//   MFMA      = v_mfma_f32_32x32x16_bf16, A = weight rows (features), B =
//               activation rows (tokens); lane l holds row l%32 and, in each
//               64-wide k step, lane half hf of MFMA j takes k = 32hf + 8j
//               .. +8 of both operands.
//   weights   = packed in MFMA tiles (wedlm_pack_weights): the 32 rows x 64
//               k of one block and step are 4 KB in the order the MFMAs read
//               them, lane l's 16 bytes of MFMA j at byte 1024j + 16l, so
//               each load instruction reads 1 KB of contiguous memory and a
//               wave's run of steps is one contiguous stretch.  Activations
//               stay row-major: lane l reads 64 contiguous bytes of its token
//               row per step (from L2).
//   output    = lane l, element e: feature 8(e/4) + 4(l/32) + e%4, token l%32.
#include <math.h>

#include <algorithm>
#include <type_traits>

#include "common.h"
#include "internal.h"
#include "wedlm_model.h"

using namespace wedlm;

namespace {

constexpr int kKStep = 64;                        // k per MFMA step (4 x 16)

// ---------------------------------------------------------------------------
// embedding: x[t] = E[token], [M] -> the mask row; fp32 residual stream
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void embed_kernel(
    const int32_t* __restrict__ tok, int mask_row, int V,
    const uint16_t* __restrict__ table, int Hd, float* __restrict__ x) {
  const int t = blockIdx.x;
  int id = tok[t];
  if (id < 0) id = mask_row;
  if (id >= V) id = mask_row;           // an id outside the table: [M]
  const u16x8_t* src =
      reinterpret_cast<const u16x8_t*>(table + static_cast<int64_t>(id) * Hd);
  float* dst = x + static_cast<int64_t>(t) * Hd;
  for (int c = threadIdx.x; c < Hd / 8; c += blockDim.x) {
    const u16x8_t v = src[c];
    floatx4_t lo, hi;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo[e] = bf16_to_f32(v[e]);
      hi[e] = bf16_to_f32(v[e + 4]);
    }
    *reinterpret_cast<floatx4_t*>(dst + c * 8) = lo;
    *reinterpret_cast<floatx4_t*>(dst + c * 8 + 4) = hi;
  }
}

// ---------------------------------------------------------------------------
// RMSNorm: y = bf16(x / sqrt(mean(x^2) + eps) * g), one workgroup per row.
// With ADD, the n_ks partial products of a split residual-add projection
// ([n_ks, M, Hd] fp32) are first added into x in split order and the sum is
// written back (the residual stream), then normalised.
// A thread owns the float4 chunks c = tid + 256 i, i < CPT, of its row and
// keeps them in registers: the loads of x, of the gain and of up to
// eight (or four) partials are all issued before the first add, so a row
// costs one memory round trip before the reduction (CPT = 0: rows longer
// than 8192, a loop over the chunks).
// ---------------------------------------------------------------------------
constexpr int kNormThreads = 256;

template <bool ADD, bool XP, int CPT>
__global__ __launch_bounds__(kNormThreads) void rmsnorm_kernel(
    float* __restrict__ x, const float* __restrict__ part, int n_ks, int M,
    const uint16_t* __restrict__ g, int Hd, float eps,
    uint16_t* __restrict__ y) {
  const int t = blockIdx.x;
  const int nc = Hd / 4;
  float* row = x + static_cast<int64_t>(t) * Hd;
  uint16_t* out = y + static_cast<int64_t>(t) * Hd;   // row-major
  auto store_out = [&](int c, const floatx4_t& v, const u16x4_t& gg, float r) {
    u16x4_t o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = f32_to_bf16(v[e] * r * bf16_to_f32(gg[e]));
    // packed (XP): the 4 values share one 16-byte chunk of a tile
    *reinterpret_cast<u16x4_t*>(XP ? y + packed_off(t, c * 4, Hd) : out + c * 4) = o;
  };
  __shared__ float wsum[kNormThreads / kWave];
  auto row_total = [&](float ss) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
    if (lane_id() == 0) wsum[threadIdx.x / kWave] = ss;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int i = 0; i < kNormThreads / kWave; ++i) tot += wsum[i];
    return 1.0f / sqrtf(tot / static_cast<float>(Hd) + eps);
  };

  if constexpr (CPT > 0) {
    // partials loaded before the first add: eight for rows of up to 4096,
    // four for longer ones (registers)
    constexpr int kNormPre = CPT <= 4 ? 8 : 4;
    floatx4_t v[CPT];
    u16x4_t gg[CPT];
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = threadIdx.x + i * kNormThreads;
      if (c < nc) {
        v[i] = *reinterpret_cast<const floatx4_t*>(row + c * 4);
        gg[i] = *reinterpret_cast<const u16x4_t*>(g + c * 4);
      }
    }
    if constexpr (ADD) {
      floatx4_t p[kNormPre][CPT];
#pragma unroll
      for (int k = 0; k < kNormPre; ++k)
        if (k < n_ks)
#pragma unroll
          for (int i = 0; i < CPT; ++i) {
            const int c = threadIdx.x + i * kNormThreads;
            if (c < nc)
              p[k][i] = *reinterpret_cast<const floatx4_t*>(
                  part + (static_cast<int64_t>(k) * M + t) * Hd + c * 4);
          }
      // split order: x + p_0 + p_1 + ...
#pragma unroll
      for (int k = 0; k < kNormPre; ++k)
        if (k < n_ks)
#pragma unroll
          for (int i = 0; i < CPT; ++i)
#pragma unroll
            for (int e = 0; e < 4; ++e) v[i][e] += p[k][i][e];
      for (int k = kNormPre; k < n_ks; ++k)
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
          const int c = threadIdx.x + i * kNormThreads;
          if (c < nc) {
            const floatx4_t q = *reinterpret_cast<const floatx4_t*>(
                part + (static_cast<int64_t>(k) * M + t) * Hd + c * 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) v[i][e] += q[e];
          }
        }
#pragma unroll
      for (int i = 0; i < CPT; ++i) {
        const int c = threadIdx.x + i * kNormThreads;
        if (c < nc) *reinterpret_cast<floatx4_t*>(row + c * 4) = v[i];
      }
    }
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = threadIdx.x + i * kNormThreads;
      if (c < nc)
        ss += v[i][0] * v[i][0] + v[i][1] * v[i][1] + v[i][2] * v[i][2] +
              v[i][3] * v[i][3];
    }
    const float r = row_total(ss);
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = threadIdx.x + i * kNormThreads;
      if (c < nc) store_out(c, v[i], gg[i], r);
    }
  } else {
    float ss = 0.f;
    for (int c = threadIdx.x; c < nc; c += kNormThreads) {
      floatx4_t v = *reinterpret_cast<const floatx4_t*>(row + c * 4);
      if constexpr (ADD) {
        for (int k = 0; k < n_ks; ++k) {
          const floatx4_t p = *reinterpret_cast<const floatx4_t*>(
              part + (static_cast<int64_t>(k) * M + t) * Hd + c * 4);
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] += p[e];
        }
        *reinterpret_cast<floatx4_t*>(row + c * 4) = v;
      }
      ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
    }
    const float r = row_total(ss);
    // every thread re-reads only the chunks it wrote itself
    for (int c = threadIdx.x; c < nc; c += kNormThreads)
      store_out(c, *reinterpret_cast<const floatx4_t*>(row + c * 4),
                *reinterpret_cast<const u16x4_t*>(g + c * 4), r);
  }
}

// ---------------------------------------------------------------------------
// per-head RMSNorm of q and k, then RoPE at the row's logical position
// (Eq. 2; "rotate half": dimension i pairs with i + D/2 at angle
// pos * theta^(-2i/D), angles in fp64); v is copied.  One workgroup per row;
// one item = 8 rotation pairs of one head (two 16-byte loads), the D/16
// items of a head sit on consecutive lanes and reduce their sum of squares
// with xor shuffles.
// PART: the q|k|v row comes as the n_ks fp32 partials of a split product
// ([n_ks, M, H*D]); they are added in split order and rounded to bf16 (the
// product's own output precision) on the way in.
// ---------------------------------------------------------------------------
constexpr int kQkThreads = 256;
constexpr int kMaxHalf = 64;

template <bool PART>
__device__ __forceinline__ u16x8_t qkv_load8(const uint16_t* x,
                                             const float* part, int64_t pstride,
                                             int n_ks, int64_t off) {
  if constexpr (!PART) {
    return *reinterpret_cast<const u16x8_t*>(x + off);
  } else {
    floatx4_t lo = *reinterpret_cast<const floatx4_t*>(part + off);
    floatx4_t hi = *reinterpret_cast<const floatx4_t*>(part + off + 4);
    for (int k = 1; k < n_ks; ++k) {
      const floatx4_t a = *reinterpret_cast<const floatx4_t*>(part + k * pstride + off);
      const floatx4_t b = *reinterpret_cast<const floatx4_t*>(part + k * pstride + off + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo[e] += a[e];
        hi[e] += b[e];
      }
    }
    u16x8_t r;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      r[e] = f32_to_bf16(lo[e]);
      r[e + 4] = f32_to_bf16(hi[e]);
    }
    return r;
  }
}

template <bool PART>
__global__ __launch_bounds__(kQkThreads) void qk_norm_rope_kernel(
    const uint16_t* __restrict__ qkv, const float* __restrict__ part,
    int n_ks, int M, const uint16_t* __restrict__ gq,
    const uint16_t* __restrict__ gk, const int32_t* __restrict__ pos_ids,
    int Hq, int Hkv, int D, double theta, float eps,
    uint16_t* __restrict__ q_out, uint16_t* __restrict__ k_out,
    uint16_t* __restrict__ v_out) {
  const int t = blockIdx.x;
  const int half = D / 2;
  const int per_head = half / 8;                  // items of a head: 4 or 8
  const int n_items = (Hq + Hkv) * per_head;
  const int H = Hq + 2 * Hkv;
  const int64_t row = static_cast<int64_t>(t) * H * D;   // element offset
  const int64_t pstride = static_cast<int64_t>(M) * H * D;
  const int nv = Hkv * D / 8;                     // 16-byte pieces of v
  // the first two rounds of q/k items and the first round of v are loaded
  // before the rotation table is computed, so its fp64 trigonometry runs
  // under their round trip
  auto load_item = [&](int it, u16x8_t& lo8, u16x8_t& hi8) {
    if (it < n_items) {
      const int head = it / per_head;
      const int j0 = (it - head * per_head) * 8;
      lo8 = qkv_load8<PART>(qkv, part, pstride, n_ks, row + head * D + j0);
      hi8 = qkv_load8<PART>(qkv, part, pstride, n_ks, row + head * D + j0 + half);
    }
  };
  u16x8_t lo0 = {}, hi0 = {}, lo1 = {}, hi1 = {}, v0 = {};
  load_item(threadIdx.x, lo0, hi0);
  load_item(threadIdx.x + kQkThreads, lo1, hi1);
  if (threadIdx.x < nv)
    v0 = qkv_load8<PART>(qkv, part, pstride, n_ks,
                         row + (Hq + Hkv) * D + threadIdx.x * 8);

  __shared__ double s_cos[kMaxHalf], s_sin[kMaxHalf];
  if (threadIdx.x < half) {
    const int j = threadIdx.x;
    const double pos = static_cast<double>(pos_ids[t]);
    const double omega = pow(theta, -2.0 * j / D);
    double sn, cs;
    sincos(pos * omega, &sn, &cs);
    s_cos[j] = cs;
    s_sin[j] = sn;
  }
  __syncthreads();
  // n_items is a multiple of per_head and every round starts at a multiple
  // of kQkThreads, so a head's items never straddle a round or a wave
  auto rotate = [&](int it, const u16x8_t& lo8, const u16x8_t& hi8) {
    const bool live = it < n_items;
    const int head = live ? it / per_head : 0;
    const int j0 = live ? (it - head * per_head) * 8 : 0;
    float a[8], b[8], ss = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      a[e] = bf16_to_f32(lo8[e]);
      b[e] = bf16_to_f32(hi8[e]);
      ss += a[e] * a[e] + b[e] * b[e];
    }
    for (int off = 1; off < per_head; off <<= 1) ss += __shfl_xor(ss, off);
    if (!live) return;
    const float r = 1.0f / sqrtf(ss / static_cast<float>(D) + eps);
    const uint16_t* g = head < Hq ? gq : gk;
    u16x8_t olo, ohi;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const double na = a[e] * r * bf16_to_f32(g[j0 + e]);
      const double nb = b[e] * r * bf16_to_f32(g[j0 + e + half]);
      const double cs = s_cos[j0 + e], sn = s_sin[j0 + e];
      olo[e] = f32_to_bf16(static_cast<float>(na * cs - nb * sn));
      ohi[e] = f32_to_bf16(static_cast<float>(nb * cs + na * sn));
    }
    uint16_t* dst = head < Hq
                        ? q_out + (static_cast<int64_t>(t) * Hq + head) * D
                        : k_out + (static_cast<int64_t>(t) * Hkv + head - Hq) * D;
    *reinterpret_cast<u16x8_t*>(dst + j0) = olo;
    *reinterpret_cast<u16x8_t*>(dst + j0 + half) = ohi;
  };
  rotate(threadIdx.x, lo0, hi0);
  if (n_items > kQkThreads) rotate(threadIdx.x + kQkThreads, lo1, hi1);
  for (int base = 2 * kQkThreads; base < n_items; base += kQkThreads) {
    u16x8_t lo8 = {}, hi8 = {};
    load_item(base + threadIdx.x, lo8, hi8);
    rotate(base + threadIdx.x, lo8, hi8);
  }
  u16x8_t* dv =
      reinterpret_cast<u16x8_t*>(v_out + static_cast<int64_t>(t) * Hkv * D);
  if (threadIdx.x < nv) dv[threadIdx.x] = v0;
  for (int e = threadIdx.x + kQkThreads; e < nv; e += kQkThreads)
    dv[e] = qkv_load8<PART>(qkv, part, pstride, n_ks, row + (Hq + Hkv) * D + e * 8);
}

// ---------------------------------------------------------------------------
// GEMM
// ---------------------------------------------------------------------------
constexpr int kGWaves = 8;
constexpr int kGThreads = kGWaves * kWave;
constexpr int kRedStride = 33;                    // LDS row of 32 tokens + 1

enum Epi { kStoreBf16 = 0, kAddF32 = 1, kSwiglu = 2 };

constexpr int kTile = 32 * kKStep;               // elements of a packed tile

struct GemmArgs {
  const uint16_t* x;      // [M, K] activations
  const uint16_t* w;      // [rows, K] weights, packed tiles
  void* out;              // [M, ldo]
  int M, N, K, ldo;
  int up_blk;             // SwiGLU: first 32-row block of the up rows
  int n_nb, n_rg;         // 32-feature blocks, row groups
  int n_ks;               // K splits over workgroups (residual add only)
  float* part;            // n_ks > 1: [n_ks, M, N] partial products
};

// XP: the SwiGLU output is written in the packed tile layout (the next
// product's input)
template <int EPI, bool XP>
__device__ __forceinline__ void gemm_store(const GemmArgs& a, int tok, int n,
                                           float g, float u) {
  const int64_t o = static_cast<int64_t>(tok) * a.ldo + n;
  if constexpr (EPI == kStoreBf16) {
    static_cast<uint16_t*>(a.out)[o] = f32_to_bf16(g);
  } else if constexpr (EPI == kAddF32) {
    static_cast<float*>(a.out)[o] += g;
  } else {
    const uint16_t r = f32_to_bf16(g / (1.0f + expf(-g)) * u);
    if constexpr (XP)
      static_cast<uint16_t*>(a.out)[packed_off(tok, n, a.N)] = r;
    else
      static_cast<uint16_t*>(a.out)[o] = r;
  }
}

// NT: weight loads carry the non-temporal hint (one row group; with several,
// the groups share the weight lines through L2).  XP: the activations come
// in the packed tile layout (ceil(M/32) tiles of 32 rows; rows past M are
// never stored), so each activation load is 1 KB of contiguous memory too;
// otherwise row-major, 64 contiguous bytes of a token row per lane and step.
// NW: waves per workgroup (8, or 4 for the split residual-add products of
// one 32-row block, whose K splits then run eight steps per wave).
template <int NB, int NA, int PF, int EPI, bool NT, bool XP, int NW>
__global__ __launch_bounds__(NW * kWave) void gemm_kernel(GemmArgs a) {
  constexpr int RB = 32 * NB;
  constexpr int TPC = 2;                            // tiles per LDS round
  constexpr int BPC = TPC / NA;                     // row blocks per round
  static_assert(NB % BPC == 0 || NB < BPC, "row blocks per round");
  static_assert(NW == 4 || NW == 8, "waves per workgroup");
  __shared__ float red[NW * TPC * 32 * kRedStride];

  // the K splits and row groups of one feature block sit on one XCD (same
  // blockIdx % 8) at neighbouring positions: the row groups share its
  // weight lines in that XCD's L2
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int per_nb = a.n_rg * a.n_ks;
  const int nb = xcd + 8 * (local / per_nb);
  const int rg = (local % per_nb) / a.n_ks;
  const int ks = local % a.n_ks;
  if (nb >= a.n_nb) return;                         // whole workgroup

  const int lane = lane_id();
  // the wave index in a scalar register: the step range and every branch on
  // it below are then uniform scalar branches
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int col = lane & 31, hf = lane >> 5;
  const int S = a.K / kKStep;
  const int k0 = ks * S / a.n_ks, k1 = (ks + 1) * S / a.n_ks;
  const int s0 = k0 + wave * (k1 - k0) / NW;
  const int s1 = k0 + (wave + 1) * (k1 - k0) / NW;
  const int n = s1 - s0;

  floatx16_t acc[NA][NB];
#pragma unroll
  for (int i = 0; i < NA; ++i)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][b][e] = 0.f;

  if (n > 0) {
    const uint16_t* wrow[NA];
#pragma unroll
    for (int i = 0; i < NA; ++i)
      wrow[i] = a.w + (static_cast<int64_t>(nb + i * a.up_blk) * S + s0) * kTile +
                lane * 8;
    const uint16_t* xrow[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if constexpr (XP) {
        const int tb = min(rg * NB + b, (a.M - 1) / 32);
        xrow[b] = a.x + (static_cast<int64_t>(tb) * S + s0) * kTile + lane * 8;
      } else {
        const int t = min(rg * RB + b * 32 + col, a.M - 1);
        xrow[b] = a.x + static_cast<int64_t>(t) * a.K + hf * 32 + s0 * kKStep;
      }
    }
    u16x8_t wa[PF][NA][4], xb[PF][NB][4];
    // every load is issued (steps past the run re-read its last step), so
    // the waits in the loop stay partial
    auto load = [&](int q, u16x8_t (&ra)[NA][4], u16x8_t (&rb)[NB][4]) {
      const int qq = min(q, n - 1);
#pragma unroll
      for (int i = 0; i < NA; ++i)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const u16x8_t* p = reinterpret_cast<const u16x8_t*>(
              wrow[i] + qq * kTile + u * 512);
          if constexpr (NT)
            ra[i][u] = __builtin_nontemporal_load(p);
          else
            ra[i][u] = *p;
        }
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int u = 0; u < 4; ++u)
          rb[b][u] = *reinterpret_cast<const u16x8_t*>(
              XP ? xrow[b] + qq * kTile + u * 512 : xrow[b] + qq * kKStep + u * 8);
    };
    auto mfma = [&](const u16x8_t (&ra)[NA][4], const u16x8_t (&rb)[NB][4]) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < NA; ++i)
#pragma unroll
          for (int b = 0; b < NB; ++b)
            acc[i][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8_t, ra[i][j]),
                __builtin_bit_cast(bf16x8_t, rb[b][j]), acc[i][b], 0, 0, 0);
    };
#pragma unroll
    for (int p = 0; p < PF; ++p) load(p, wa[p], xb[p]);
    // whole groups of PF steps with no branch inside; step q + u sits in
    // stage u, so the last n % PF steps are in stages 0 .. n % PF - 1
    int q = 0;
    for (; q + PF <= n; q += PF) {
#pragma unroll
      for (int u = 0; u < PF; ++u) {
        mfma(wa[u], xb[u]);
        load(q + u + PF, wa[u], xb[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < PF - 1; ++u)
      if (q + u < n) mfma(wa[u], xb[u]);
  }

  // sum the NW waves' partial tiles in wave order, TPC tiles per round
  constexpr int kRounds = (NA * NB + TPC - 1) / TPC;
#pragma unroll
  for (int rd = 0; rd < kRounds; ++rd) {
    if (rd > 0) __syncthreads();
#pragma unroll
    for (int tt = 0; tt < TPC; ++tt) {
      const int tile = rd * TPC + tt;               // = b * NA + i
      if (tile >= NA * NB) break;
      const int i = tile % NA, b = tile / NA;
      float* dst = red + (wave * TPC + tt) * 32 * kRedStride;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int f = 8 * (e >> 2) + 4 * hf + (e & 3);
        dst[f * kRedStride + col] = acc[i][b][e];
      }
    }
    __syncthreads();
    // thread -> (feature f, token t): 32 features x 2 NW tokens per pass
    const int f = threadIdx.x & 31;
#pragma unroll
    for (int half = 0; half < 16 / NW; ++half) {
      const int tl = (threadIdx.x >> 5) + 2 * NW * half;
#pragma unroll
      for (int bb = 0; bb < BPC; ++bb) {
        const int tile0 = rd * TPC + bb * NA;
        if (tile0 >= NA * NB) break;
        const int b = tile0 / NA;
        const int tok = rg * RB + b * 32 + tl;
        float v[NA];
#pragma unroll
        for (int i = 0; i < NA; ++i) {
          float s = 0.f;
#pragma unroll
          for (int w = 0; w < NW; ++w)
            s += red[((w * TPC + bb * NA + i) * 32 + f) * kRedStride + tl];
          v[i] = s;
        }
        if (tok >= a.M) continue;
        if (a.n_ks == 1) {
          gemm_store<EPI, XP>(a, tok, nb * 32 + f, v[0], v[NA - 1]);
        } else {
          // split K (residual add): this split's partial, summed into the
          // residual stream later in split order
          a.part[(static_cast<int64_t>(ks) * a.M + tok) * a.N + nb * 32 + f] =
              v[0];
        }
      }
    }
  }
}

// x[t][n] += sum over splits k (in order) of part[k][t][n]
__global__ __launch_bounds__(256) void add_partials_kernel(
    float* __restrict__ x, int ldx, const float* __restrict__ part, int n_ks,
    int M, int N) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= static_cast<int64_t>(M) * N) return;
  const int t = static_cast<int>(i / N), n = static_cast<int>(i % N);
  float v = x[static_cast<int64_t>(t) * ldx + n];
  for (int k = 0; k < n_ks; ++k) v += part[static_cast<int64_t>(k) * M * N + i];
  x[static_cast<int64_t>(t) * ldx + n] = v;
}

// ---------------------------------------------------------------------------
// 2-D tiled GEMM for many window rows (M >= 128: batches of windows).  A
// workgroup computes 256 features (8 blocks; for SwiGLU 4 gate blocks and
// their 4 up blocks) x 128 tokens (4 row tiles) over its run of K steps.
// Per 64-wide step the 12 packed 4 KB tiles (8 weight, 4 activation) go
// from HBM into LDS as they are, with LDS-destination buffer loads (the
// packed layout is already the MFMA operand order, so every fragment read
// is 16 contiguous bytes per lane and no register holds a tile in
// transit); each of the 8 waves computes a 64 x 64 piece (2 feature blocks
// x 2 row tiles, 16 MFMAs per step), so every LDS byte a wave reads feeds
// two MFMAs.  A ring of three LDS stages: the tiles of step s+2 load while
// step s computes, one barrier per step.  Activations must be packed
// (ceil(M/32) tiles).
// ---------------------------------------------------------------------------
constexpr int k2dFeat = 8;                        // feature blocks per WG
constexpr int k2dTok = 4;                         // row tiles per WG
constexpr int k2dTiles = k2dFeat + k2dTok;        // 12 tiles per step
constexpr int k2dStage = k2dTiles * kTile * 2;    // 48 KB per LDS buffer
constexpr int k2dChunks = k2dTiles * 4 / kGWaves;       // 1 KB chunks per wave: 6
constexpr int k2dStages = 3;                      // LDS ring: 144 KB

struct Gemm2dArgs {
  const uint16_t* x;      // packed activations, ceil(M/32) row tiles
  const uint16_t* w;      // packed weights
  void* out;
  float* part;            // n_ks > 1 (residual add, stored q|k|v): [n_ks, M, N]
  int M, N, K, ldo;
  int n_fb;               // 32-feature blocks of the output (N / 32)
  int n_ft, n_tt, n_ks;   // feature tiles, row tiles, K splits
};

template <int EPI>
__global__ __launch_bounds__(kGThreads) void gemm2d_kernel(Gemm2dArgs a) {
  __shared__ __attribute__((aligned(1024))) char lds2[k2dStages * k2dStage];
  // tile order: the K splits and row tiles of one feature tile on one XCD
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int per_ft = a.n_tt * a.n_ks;
  const int ft = xcd + 8 * (local / per_ft);
  const int tt = (local % per_ft) / a.n_ks;
  const int ks = local % a.n_ks;
  if (ft >= a.n_ft) return;                          // whole workgroup

  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int S = a.K / kKStep;
  const int s0 = ks * S / a.n_ks, s1 = (ks + 1) * S / a.n_ks;
  const int n = s1 - s0;                             // >= 1 (plan)
  const int last_rt = (a.M - 1) / 32;

  // weight block of LDS tile i (0..7): consecutive feature blocks, or for
  // SwiGLU gate blocks 0..3 then their up blocks (clamped at the end: those
  // outputs are never stored)
  const int out_blocks = EPI == kSwiglu ? k2dFeat / 2 : k2dFeat;
  auto wblock = [&](int i) {
    const int f = ft * out_blocks + (EPI == kSwiglu ? (i & 3) : i);
    const int fc = min(f, a.n_fb - 1);
    return (EPI == kSwiglu && i >= 4) ? fc + a.n_fb : fc;
  };
  // The 48 KB of a step go straight from HBM into its LDS stage: wave w
  // moves the 1 KB chunks c = 6w .. 6w+5 (tile c / 4, MFMA j = c % 4), one
  // load instruction each, lane l's 16 bytes landing at byte 16 l of the
  // chunk, which is where the packed layout already keeps them.  Each chunk
  // is read through a buffer resource over its tile's run of steps.
  const uint32_t lds0 =
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_t*)lds2));
  i32x4_t rs[k2dChunks];
#pragma unroll
  for (int u = 0; u < k2dChunks; ++u) {
    const int tile = (wave * k2dChunks + u) >> 2;
    const int64_t blk = tile < k2dFeat ? wblock(tile)
                                       : min(tt * k2dTok + tile - k2dFeat, last_rt);
    rs[u] = buffer_rsrc((tile < k2dFeat ? a.w : a.x) + (blk * S + s0) * kTile,
                        n * kTile * 2);
  }
  auto issue = [&](int q, int stage) {
    const int qq = min(q, n - 1);                    // past the run: re-read
#pragma unroll
    for (int u = 0; u < k2dChunks; ++u) {
      const int c = wave * k2dChunks + u;
      load_to_lds16<false>(
          rs[u], qq * kTile * 2 + (c & 3) * 1024 + lane * 16,
          __builtin_amdgcn_readfirstlane(lds0 + stage * k2dStage + c * 1024));
    }
  };
  // wave tile: feature blocks fb0, fb0+1 (SwiGLU: gate fw and up fw + 4) x
  // row tiles 2*tw, 2*tw+1 of the workgroup
  const int fw = wave & 3, tw = wave >> 2;
  const int fa = EPI == kSwiglu ? fw : 2 * fw;
  const int fb = EPI == kSwiglu ? fw + 4 : 2 * fw + 1;
  floatx16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  auto compute = [&](int buf) {
    const char* base = lds2 + buf * k2dStage + lane * 16;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bf16x8_t a0 = *reinterpret_cast<const bf16x8_t*>(base + fa * 4096 + j * 1024);
      const bf16x8_t a1 = *reinterpret_cast<const bf16x8_t*>(base + fb * 4096 + j * 1024);
      const bf16x8_t b0 = *reinterpret_cast<const bf16x8_t*>(
          base + (k2dFeat + 2 * tw) * 4096 + j * 1024);
      const bf16x8_t b1 = *reinterpret_cast<const bf16x8_t*>(
          base + (k2dFeat + 2 * tw + 1) * 4096 + j * 1024);
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
    }
  };

  // step q computes from stage q % 3 while the loads of step q+2 fill stage
  // (q+2) % 3, read last in step q-1 (before the barrier that ended it);
  // before the barrier that ends step q every wave waits for its loads of
  // step q+1, leaving only those of q+2 in flight.
  issue(0, 0);
  issue(1, 1);
  wait_vmcnt<k2dChunks>();
  __syncthreads();
  for (int q = 0; q < n; ++q) {
    issue(q + 2, (q + 2) % k2dStages);
    compute(q % k2dStages);
    wait_vmcnt<k2dChunks>();
    __syncthreads();
  }
  wait_vmcnt<0>();   // surplus re-reads retire before the workgroup ends

  // epilogue from registers: lane l, element e = 4g + r is feature
  // 8g + 4(l/32) + r of its block and token l%32 of its row tile, so the 4
  // values of a group are 4 consecutive features of one token
  const int hf = lane >> 5, col = lane & 31;
#pragma unroll
  for (int tj = 0; tj < 2; ++tj) {
    const int tok = (tt * k2dTok + 2 * tw + tj) * 32 + col;
    if (tok >= a.M) continue;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      if constexpr (EPI == kSwiglu) {
        const int f = (ft * (k2dFeat / 2) + fw) * 32 + 8 * g + 4 * hf;
        if (f >= a.N) continue;
        u16x4_t o;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float gg = acc[0][tj][4 * g + r], uu = acc[1][tj][4 * g + r];
          o[r] = f32_to_bf16(gg / (1.0f + expf(-gg)) * uu);
        }
        *reinterpret_cast<u16x4_t*>(static_cast<uint16_t*>(a.out) +
                                    packed_off(tok, f, a.N)) = o;
      } else {
#pragma unroll
        for (int fi = 0; fi < 2; ++fi) {
          const int f = (ft * k2dFeat + (fi ? fb : fa)) * 32 + 8 * g + 4 * hf;
          if (f >= a.N) continue;
          floatx4_t v;
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] = acc[fi][tj][4 * g + r];
          const int64_t o = static_cast<int64_t>(tok) * a.ldo + f;
          if (EPI == kStoreBf16 && a.n_ks == 1) {
            u16x4_t h;
#pragma unroll
            for (int r = 0; r < 4; ++r) h[r] = f32_to_bf16(v[r]);
            *reinterpret_cast<u16x4_t*>(static_cast<uint16_t*>(a.out) + o) = h;
          } else if (EPI == kAddF32 && a.n_ks == 1) {
            floatx4_t* p = reinterpret_cast<floatx4_t*>(static_cast<float*>(a.out) + o);
            const floatx4_t old = *p;
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] += old[r];
            *p = v;
          } else {
            *reinterpret_cast<floatx4_t*>(
                a.part + (static_cast<int64_t>(ks) * a.M + tok) * a.N + f) = v;
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Wide SwiGLU tiles for large grids: a workgroup computes 128 features
// (gate blocks 0..3 and their up blocks) x 256 tokens (8 row tiles) over
// the whole K.  Wave w takes gate block w%4 and its up block x row tiles
// 4(w/4) .. 4(w/4)+3: each A fragment read from LDS feeds four MFMAs and
// each B fragment two, 0.75 KB of LDS reads per MFMA against 1 KB in the
// kernel above.  Per step the 16 packed tiles (64 KB) go to LDS as there;
// a ring of two stages (128 KB): the tiles of step s+1 load while step s
// computes.  Each output element sums its k steps in the same order as the
// kernel above, so the two give the same bits.  Used when its grid fills
// most of the chip (at 512 rows and 12288 features: 92-99 against 109-127
// us); on smaller grids the 128-token tiles are faster.
// ---------------------------------------------------------------------------
constexpr int kWTok = 8;                          // row tiles per WG
constexpr int kWTiles = k2dFeat + kWTok;          // 16 tiles per step
constexpr int kWStage = kWTiles * kTile * 2;      // 64 KB per LDS buffer
constexpr int kWChunks = kWTiles * 4 / kGWaves;   // 1 KB chunks per wave: 8
constexpr int kWStages = 2;                       // LDS ring: 128 KB

__global__ __launch_bounds__(kGThreads) void gemm2d_swiglu_wide_kernel(
    Gemm2dArgs a) {
  __shared__ __attribute__((aligned(1024))) char lds2[kWStages * kWStage];
  // tile order: the row tiles of one feature tile on one XCD
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int ft = xcd + 8 * (local / a.n_tt);
  const int tt = local % a.n_tt;
  if (ft >= a.n_ft) return;                          // whole workgroup

  const int lane = lane_id();
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int n = a.K / kKStep;
  const int last_rt = (a.M - 1) / 32;
  // gate blocks 0..3 then their up blocks (clamped at the end: those
  // outputs are never stored)
  auto wblock = [&](int i) {
    const int f = ft * (k2dFeat / 2) + (i & 3);
    const int fc = min(f, a.n_fb - 1);
    return i >= 4 ? fc + a.n_fb : fc;
  };
  // wave w moves the 1 KB chunks c = 8w .. 8w+7 (tile c / 4, MFMA c % 4)
  const uint32_t lds0 =
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_t*)lds2));
  i32x4_t rs[kWChunks];
#pragma unroll
  for (int u = 0; u < kWChunks; ++u) {
    const int tile = (wave * kWChunks + u) >> 2;
    const int64_t blk = tile < k2dFeat
                            ? wblock(tile)
                            : min(tt * kWTok + tile - k2dFeat, last_rt);
    rs[u] = buffer_rsrc((tile < k2dFeat ? a.w : a.x) + blk * n * kTile,
                        n * kTile * 2);
  }
  auto issue = [&](int q, int stage) {
    const int qq = min(q, n - 1);                    // past the run: re-read
#pragma unroll
    for (int u = 0; u < kWChunks; ++u) {
      const int c = wave * kWChunks + u;
      load_to_lds16<false>(
          rs[u], qq * kTile * 2 + (c & 3) * 1024 + lane * 16,
          __builtin_amdgcn_readfirstlane(lds0 + stage * kWStage + c * 1024));
    }
  };
  const int fw = wave & 3, tw = wave >> 2;
  floatx16_t acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  auto compute = [&](int buf) {
    const char* base = lds2 + buf * kWStage + lane * 16;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bf16x8_t a0 =
          *reinterpret_cast<const bf16x8_t*>(base + fw * 4096 + j * 1024);
      const bf16x8_t a1 = *reinterpret_cast<const bf16x8_t*>(
          base + (fw + 4) * 4096 + j * 1024);
      bf16x8_t b[4];
#pragma unroll
      for (int t = 0; t < 4; ++t)
        b[t] = *reinterpret_cast<const bf16x8_t*>(
            base + (k2dFeat + 4 * tw + t) * 4096 + j * 1024);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        acc[0][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b[t], acc[0][t], 0, 0, 0);
        acc[1][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b[t], acc[1][t], 0, 0, 0);
      }
    }
  };

  // step q computes from stage q % 2 while the loads of step q+1 fill the
  // other stage, read last in step q-1 (before the barrier that ended it);
  // before the barrier that ends step q every wave waits for its loads.
  issue(0, 0);
  wait_vmcnt<0>();
  __syncthreads();
  for (int q = 0; q < n; ++q) {
    issue(q + 1, (q + 1) & 1);
    compute(q & 1);
    wait_vmcnt<0>();
    __syncthreads();
  }

  // epilogue as in gemm2d_kernel (lane l, element 4g + r: feature
  // 8g + 4(l/32) + r of its block, token l%32 of its row tile)
  const int hf = lane >> 5, col = lane & 31;
#pragma unroll
  for (int tj = 0; tj < 4; ++tj) {
    const int tok = (tt * kWTok + 4 * tw + tj) * 32 + col;
    if (tok >= a.M) continue;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int f = (ft * (k2dFeat / 2) + fw) * 32 + 8 * g + 4 * hf;
      if (f >= a.N) continue;
      u16x4_t o;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float gg = acc[0][tj][4 * g + r], uu = acc[1][tj][4 * g + r];
        o[r] = f32_to_bf16(gg / (1.0f + expf(-gg)) * uu);
      }
      *reinterpret_cast<u16x4_t*>(static_cast<uint16_t*>(a.out) +
                                  packed_off(tok, f, a.N)) = o;
    }
  }
}

// out[t][n] (bf16) = sum over splits k (in order) of part[k][t][n], four
// consecutive n per thread (N a multiple of 32, ldo of 4)
__global__ __launch_bounds__(256) void sum_partials_bf16_kernel(
    uint16_t* __restrict__ out, int ldo, const float* __restrict__ part,
    int n_ks, int M, int N) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t n4 = N / 4;
  if (i >= static_cast<int64_t>(M) * n4) return;
  const int64_t t = i / n4;
  const int n = static_cast<int>(i % n4) * 4;
  floatx4_t v = {0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < n_ks; ++k) {
    const floatx4_t p = *reinterpret_cast<const floatx4_t*>(
        part + (static_cast<int64_t>(k) * M + t) * N + n);
#pragma unroll
    for (int r = 0; r < 4; ++r) v[r] += p[r];
  }
  u16x4_t h;
#pragma unroll
  for (int r = 0; r < 4; ++r) h[r] = f32_to_bf16(v[r]);
  *reinterpret_cast<u16x4_t*>(out + t * ldo + n) = h;
}

// row-major [rows, K] -> packed MFMA tiles; one thread moves 16 bytes and
// the writes are contiguous
__global__ __launch_bounds__(256) void pack_kernel(
    const uint16_t* __restrict__ w, int K, int64_t n_chunks,
    uint16_t* __restrict__ packed) {
  const int64_t c = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (c >= n_chunks) return;
  const int S = K / kKStep;
  const int64_t tile = c >> 8;                     // 256 chunks per tile
  const int idx = static_cast<int>(c & 255);
  const int u = idx >> 6, l = idx & 63;
  const int64_t rb = tile / S;
  const int s = static_cast<int>(tile - rb * S);
  const int64_t row = rb * 32 + (l & 31);
  const int k = s * kKStep + (l >> 5) * 32 + u * 8;
  *reinterpret_cast<u16x8_t*>(packed + c * 8) =
      *reinterpret_cast<const u16x8_t*>(w + row * K + k);
}

// rows per group: 32, 64, then 128 (64 for SwiGLU, two weight blocks)
int gemm_nb(int M, bool swiglu) {
  if (M <= 32) return 1;
  if (M <= 64 || swiglu) return 2;
  return 4;
}

// the largest row block of each kernel family also serves several row
// groups; the smaller ones only ever run as one
template <int NB, int NA, int PF, int EPI, bool XP, int NW = kGWaves>
void gemm_launch_xp(const GemmArgs& a, hipStream_t st) {
  const int64_t grid = 8ll * a.n_rg * a.n_ks * ((a.n_nb + 7) / 8);
  if constexpr (NB * NA == 4) {
    if (a.n_rg > 1) {
      hipLaunchKernelGGL((gemm_kernel<NB, NA, PF, EPI, false, XP, NW>),
                         dim3(grid), dim3(NW * kWave), 0, st, a);
      return;
    }
  }
  hipLaunchKernelGGL((gemm_kernel<NB, NA, PF, EPI, true, XP, NW>), dim3(grid),
                     dim3(NW * kWave), 0, st, a);
}

template <int NB, int NA, int PF, int EPI, int NW = kGWaves>
void gemm_launch(const GemmArgs& a, bool xp, hipStream_t st) {
  if (xp) gemm_launch_xp<NB, NA, PF, EPI, true, NW>(a, st);
  else gemm_launch_xp<NB, NA, PF, EPI, false, NW>(a, st);
}

bool gemm_shape_ok(int M, int N, int K) {
  return M >= 1 && N >= 32 && N % 32 == 0 && K >= kKStep && K % kKStep == 0 &&
         static_cast<int64_t>(M) * K < (1ll << 40) &&
         static_cast<int64_t>(N) * K * 2 < (1ll << 40);
}

size_t up256(size_t v) { return (v + 255) & ~static_cast<size_t>(255); }

// The plan of one product: row block, row groups and K splits.  A residual-
// add product (N = hidden: few feature blocks), and the q|k|v product when
// its caller sums the partials (split_store), split K over workgroups until
// about one workgroup per CU streams weights, never below one step per wave;
// the splits write fp32 partials ([n_ks, M, N]) that the next RMSNorm (or,
// standing alone, add_partials_kernel), or the q/k norm, sums in split
// order.  No workgroup waits for another.
struct GemmPlan {
  int nb, n_nb, n_rg, n_ks;
  int nw;                 // waves per workgroup of the split-K kernel
  bool two_d;             // the 2-D tiled kernel (packed activations, many rows)
  bool wide;              // its 256-token SwiGLU tiles
  int n_ft, n_tt;         // its feature and row tiles
  size_t part_bytes;
};

// window rows from which packed activations go through the 2-D kernel (at
// 128 rows the split-K kernel is faster: 8.1 against 9.9 ms per 36-layer
// step)
constexpr int k2dMinRows = 256;

// workgroups a split product aims at: about one per CU (with few rows, 512
// and 768 made the 36-layer step at B = 1 slower: 5.00 -> 5.29 and 5.91 ms)
constexpr int kGemmTargetWgs = 256;
// the wide SwiGLU tiles from this many workgroups (three quarters of the
// CUs; at 96 or 128 workgroups the 128-token tiles measured faster)
constexpr int kWideMinWgs = 3 * kGemmTargetWgs / 4;

GemmPlan gemm_plan(int M, int N, int K, int epi, bool xp = false,
                   bool split_store = false) {
  GemmPlan p{};
  if (xp && M >= k2dMinRows) {
    // 2-D tiles; a residual-add product with few tiles splits K (at least
    // four steps per split)
    p.two_d = true;
    p.n_nb = N / 32;
    p.n_ft = (p.n_nb + (epi == kSwiglu ? 3 : 7)) / (epi == kSwiglu ? 4 : 8);
    p.n_tt = (M + 32 * k2dTok - 1) / (32 * k2dTok);
    p.n_ks = 1;
    if (epi == kSwiglu) {
      const int n_tt_w = (M + 32 * kWTok - 1) / (32 * kWTok);
      if (p.n_ft * n_tt_w >= kWideMinWgs) {
        p.wide = true;
        p.n_tt = n_tt_w;
      }
    }
    // a stored product (q|k|v) with few tiles splits K too; its fp32
    // partials are summed into bf16 right after
    if (epi == kAddF32 || epi == kStoreBf16)
      p.n_ks = std::max(1, std::min(kGemmTargetWgs / (p.n_ft * p.n_tt),
                                    K / kKStep / 4));
    if (p.n_ks > 1)
      p.part_bytes = static_cast<size_t>(p.n_ks) * M * N * sizeof(float);
    return p;
  }
  p.nb = gemm_nb(M, epi == kSwiglu);
  p.n_nb = N / 32;
  p.n_rg = (M + 32 * p.nb - 1) / (32 * p.nb);
  p.n_ks = 1;
  p.nw = kGWaves;
  if (epi == kAddF32 && p.nb == 1 && K / kKStep <= 64) {
    // one 32-row block and K up to 4096: four-wave workgroups, K split so
    // that a wave runs about eight steps (at the o product's 4096 x 4096,
    // 11.0 -> 9.6 us).  Longer K keeps eight waves and two splits: the down
    // product split six ways this way took 24.1 against 23.0 us, and its
    // RMSNorm then adds six partials
    p.nw = 4;
    p.n_ks = std::max(1, K / kKStep / (4 * 8));
  } else if (epi == kAddF32 || (epi == kStoreBf16 && split_store)) {
    const int wgs = p.n_nb * p.n_rg;
    p.n_ks = std::max(1, std::min(kGemmTargetWgs / wgs, K / kKStep / kGWaves));
  }
  if (p.n_ks > 1)
    p.part_bytes = static_cast<size_t>(p.n_ks) * M * N * sizeof(float);
  return p;
}

// Launches the product; with K split, the partials go to `part` and the
// caller adds them (defer) or add_partials_kernel does right after.
// xp: x (and a SwiGLU output) in the packed tile layout
int gemm(const uint16_t* x, const uint16_t* w, int M, int N, int K, void* out,
         int ldo, int epi, void* part, size_t part_bytes, bool defer, bool xp,
         hipStream_t st, int* n_ks_out = nullptr) {
  if (!x || !w || !out) return WEDLM_E_ARG;
  if (epi != kStoreBf16 && epi != kAddF32 && epi != kSwiglu) return WEDLM_E_ARG;
  if (!gemm_shape_ok(M, N, K) || ldo < N) return WEDLM_E_SHAPE;
  const GemmPlan p = gemm_plan(M, N, K, epi, xp, defer);
  if (p.part_bytes > 0 && (!part || part_bytes < p.part_bytes))
    return WEDLM_E_WORKSPACE;
  if (p.two_d) {
    if ((epi == kSwiglu && N % 32 != 0) || ldo % 4 != 0) return WEDLM_E_SHAPE;
    Gemm2dArgs g{};
    g.x = x; g.w = w; g.out = out; g.part = static_cast<float*>(part);
    g.M = M; g.N = N; g.K = K; g.ldo = ldo;
    g.n_fb = p.n_nb; g.n_ft = p.n_ft; g.n_tt = p.n_tt; g.n_ks = p.n_ks;
    const int64_t grid = 8ll * p.n_tt * p.n_ks * ((p.n_ft + 7) / 8);
    if (grid > (1ll << 30)) return WEDLM_E_SHAPE;
    if (p.wide)
      hipLaunchKernelGGL(gemm2d_swiglu_wide_kernel, dim3(grid),
                         dim3(kGThreads), 0, st, g);
    else if (epi == kSwiglu)
      hipLaunchKernelGGL(gemm2d_kernel<kSwiglu>, dim3(grid), dim3(kGThreads),
                         0, st, g);
    else if (epi == kAddF32)
      hipLaunchKernelGGL(gemm2d_kernel<kAddF32>, dim3(grid), dim3(kGThreads),
                         0, st, g);
    else
      hipLaunchKernelGGL(gemm2d_kernel<kStoreBf16>, dim3(grid),
                         dim3(kGThreads), 0, st, g);
    WEDLM_LAUNCH_CHECK();
    if (n_ks_out) *n_ks_out = p.n_ks;
    if (p.n_ks > 1 && epi == kStoreBf16 && !defer) {
      const int64_t total4 = static_cast<int64_t>(M) * (N / 4);
      hipLaunchKernelGGL(sum_partials_bf16_kernel, dim3((total4 + 255) / 256),
                         dim3(256), 0, st, static_cast<uint16_t*>(out), ldo,
                         g.part, p.n_ks, M, N);
      WEDLM_LAUNCH_CHECK();
    } else if (p.n_ks > 1 && !defer) {
      const int64_t total = static_cast<int64_t>(M) * N;
      hipLaunchKernelGGL(add_partials_kernel, dim3((total + 255) / 256),
                         dim3(256), 0, st, static_cast<float*>(out), ldo,
                         g.part, p.n_ks, M, N);
      WEDLM_LAUNCH_CHECK();
    }
    return WEDLM_OK;
  }
  GemmArgs a{};
  a.x = x; a.w = w; a.out = out; a.M = M; a.N = N; a.K = K; a.ldo = ldo;
  a.up_blk = N / 32;
  a.n_nb = p.n_nb;
  a.n_rg = p.n_rg;
  a.n_ks = p.n_ks;
  a.part = static_cast<float*>(part);
  if (8ll * a.n_rg * a.n_ks * ((a.n_nb + 7) / 8) > (1ll << 30))
    return WEDLM_E_SHAPE;
  const int nb = p.nb;
  if (epi == kSwiglu) {
    if (nb == 1) gemm_launch<1, 2, 2, kSwiglu>(a, xp, st);
    else gemm_launch<2, 2, 2, kSwiglu>(a, xp, st);
  } else if (epi == kAddF32) {
    if (nb == 1 && p.nw == 4) gemm_launch<1, 1, 4, kAddF32, 4>(a, xp, st);
    else if (nb == 1) gemm_launch<1, 1, 4, kAddF32>(a, xp, st);
    else if (nb == 2) gemm_launch<2, 1, 2, kAddF32>(a, xp, st);
    else gemm_launch<4, 1, 2, kAddF32>(a, xp, st);
  } else {
    if (nb == 1) gemm_launch<1, 1, 4, kStoreBf16>(a, xp, st);
    else if (nb == 2) gemm_launch<2, 1, 2, kStoreBf16>(a, xp, st);
    else gemm_launch<4, 1, 2, kStoreBf16>(a, xp, st);
  }
  WEDLM_LAUNCH_CHECK();
  if (n_ks_out) *n_ks_out = p.n_ks;
  if (p.n_ks > 1 && !defer) {
    const int64_t total = static_cast<int64_t>(M) * N;
    hipLaunchKernelGGL(add_partials_kernel, dim3((total + 255) / 256),
                       dim3(256), 0, st, static_cast<float*>(out), ldo,
                       a.part, p.n_ks, M, N);
    WEDLM_LAUNCH_CHECK();
  }
  return WEDLM_OK;
}

// RMSNorm of the residual stream, first adding pending split partials; xp:
// y in the packed tile layout (Hd a multiple of 64)
int norm(float* x, const float* part, int n_ks, int M, int Hd,
         const uint16_t* g, float eps, uint16_t* y, bool xp, hipStream_t st) {
  const bool add = part && n_ks > 1;
  const int nc = Hd / 4;
  const int cpt = nc <= kNormThreads ? 1 : nc <= 2 * kNormThreads ? 2
                  : nc <= 4 * kNormThreads ? 4 : nc <= 8 * kNormThreads ? 8 : 0;
  using K = void (*)(float*, const float*, int, int, const uint16_t*, int,
                     float, uint16_t*);
  auto pick = [&](auto tag) -> K {
    constexpr int C = decltype(tag)::value;
    return add ? (xp ? rmsnorm_kernel<true, true, C> : rmsnorm_kernel<true, false, C>)
               : (xp ? rmsnorm_kernel<false, true, C> : rmsnorm_kernel<false, false, C>);
  };
  const K k = cpt == 1   ? pick(std::integral_constant<int, 1>{})
              : cpt == 2 ? pick(std::integral_constant<int, 2>{})
              : cpt == 4 ? pick(std::integral_constant<int, 4>{})
              : cpt == 8 ? pick(std::integral_constant<int, 8>{})
                         : pick(std::integral_constant<int, 0>{});
  hipLaunchKernelGGL(k, dim3(M), dim3(kNormThreads), 0, st, x,
                     add ? part : nullptr, add ? n_ks : 0, M, g, Hd, eps, y);
  WEDLM_LAUNCH_CHECK();
  return WEDLM_OK;
}

// q/k RMSNorm + RoPE of M rows; part: the n_ks > 1 split partials of the
// q|k|v product instead of its bf16 output
int qk_norm_rope(const uint16_t* qkv, const float* part, int n_ks, int M,
                 const uint16_t* gq, const uint16_t* gk, const int32_t* pos,
                 int Hq, int Hkv, int D, double theta, float eps,
                 uint16_t* q_out, uint16_t* k_out, uint16_t* v_out,
                 hipStream_t st) {
  if (part && n_ks > 1)
    hipLaunchKernelGGL(qk_norm_rope_kernel<true>, dim3(M), dim3(kQkThreads), 0,
                       st, qkv, part, n_ks, M, gq, gk, pos, Hq, Hkv, D, theta,
                       eps, q_out, k_out, v_out);
  else
    hipLaunchKernelGGL(qk_norm_rope_kernel<false>, dim3(M), dim3(kQkThreads), 0,
                       st, qkv, part, 1, M, gq, gk, pos, Hq, Hkv, D, theta,
                       eps, q_out, k_out, v_out);
  WEDLM_LAUNCH_CHECK();
  return WEDLM_OK;
}

bool config_ok(const wedlm_model_config* c) {
  return c && c->n_layers >= 1 && c->hidden >= 256 && c->hidden % 256 == 0 &&
         c->n_kv_heads >= 1 && c->n_heads % c->n_kv_heads == 0 &&
         (c->head_dim == 64 || c->head_dim == 128) && c->inter >= 32 &&
         c->inter % 64 == 0 && c->vocab >= 1 && c->mask_token >= 0 &&
         c->mask_token < c->vocab && c->rope_theta > 1.0 && c->rms_eps > 0.f &&
         (static_cast<int64_t>(c->n_heads) * c->head_dim) % kKStep == 0;
}

// workspace carve-up of the forward, 256-byte aligned pieces
struct Carve {
  size_t part, x, xn, qkv, q, attn, act, attn_ws, lm_ws, total;
  size_t part_bytes;
};


Carve carve(const wedlm_model_config* c, int B, int W, int max_prefix_len) {
  const size_t M = static_cast<size_t>(B) * W;
  const size_t Hd = c->hidden, D = c->head_dim;
  const size_t Hq = c->n_heads, Hkv = c->n_kv_heads;
  Carve k{};
  size_t off = 0;
  // split partials of the two residual-add products (each is summed by the
  // next RMSNorm before the other is written)
  const int Mi = static_cast<int>(M);
  // and of the q|k|v product (summed by the q/k norm that reads it)
  k.part_bytes = std::max(
      std::max(gemm_plan(Mi, c->hidden, c->n_heads * c->head_dim, kAddF32, true)
                   .part_bytes,
               gemm_plan(Mi, c->hidden, c->inter, kAddF32, true).part_bytes),
      gemm_plan(Mi, (c->n_heads + 2 * c->n_kv_heads) * c->head_dim, c->hidden,
                kStoreBf16, true, true).part_bytes);
  k.part = off; off += up256(k.part_bytes);
  k.x = off;    off += up256(M * Hd * 4);
  const size_t Mp = (M + 31) / 32 * 32;           // packed: whole tiles
  k.xn = off;   off += up256(Mp * Hd * 2);
  k.qkv = off;  off += up256(M * (Hq + 2 * Hkv) * D * 2);
  k.q = off;    off += up256(M * Hq * D * 2);
  k.attn = off; off += up256(Mp * Hq * D * 2);   // packed tiles
  k.act = off;  off += up256(Mp * c->inter * 2);
  k.attn_ws = off;
  off += up256(wedlm_window_attn_workspace_size(B, W, c->n_heads,
                                                c->n_kv_heads, c->head_dim,
                                                max_prefix_len));
  k.lm_ws = off;
  off += up256(wedlm_lm_head_score_workspace_size(static_cast<int32_t>(M),
                                                  c->hidden, c->vocab));
  k.total = off;
  return k;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------

extern "C" int wedlm_embed(const int32_t* tok, int32_t M, int32_t mask_token,
                           const uint16_t* table, int32_t V, int32_t Hd,
                           float* x, void* stream) {
  if (!tok || !table || !x) return WEDLM_E_ARG;
  if (M < 1 || V < 1 || mask_token < 0 || mask_token >= V || Hd < 8 ||
      Hd % 8 != 0)
    return WEDLM_E_SHAPE;
  hipLaunchKernelGGL(embed_kernel, dim3(M), dim3(256), 0,
                     static_cast<hipStream_t>(stream), tok, mask_token, V,
                     table, Hd, x);
  WEDLM_LAUNCH_CHECK();
  return WEDLM_OK;
}

extern "C" int wedlm_rmsnorm(const float* x, const uint16_t* gain, int32_t M,
                             int32_t Hd, float eps, uint16_t* y,
                             void* stream) {
  if (!x || !gain || !y || !(eps > 0.f)) return WEDLM_E_ARG;
  if (M < 1 || Hd < 4 || Hd % 4 != 0) return WEDLM_E_SHAPE;
  // without partials the kernel only reads x
  return norm(const_cast<float*>(x), nullptr, 0, M, Hd, gain, eps, y, false,
              static_cast<hipStream_t>(stream));
}

extern "C" int wedlm_pack_weights(const uint16_t* w, int64_t rows, int32_t K,
                                  uint16_t* packed, void* stream) {
  if (!w || !packed) return WEDLM_E_ARG;
  if (rows < 32 || rows % 32 != 0 || K < kKStep || K % kKStep != 0)
    return WEDLM_E_SHAPE;
  const int64_t n_chunks = rows * K / 8;
  const int64_t grid = (n_chunks + 255) / 256;
  if (grid > 0x7fffffffll) return WEDLM_E_SHAPE;
  hipLaunchKernelGGL(pack_kernel, dim3(static_cast<unsigned>(grid)), dim3(256),
                     0, static_cast<hipStream_t>(stream), w, K, n_chunks,
                     packed);
  WEDLM_LAUNCH_CHECK();
  return WEDLM_OK;
}

extern "C" size_t wedlm_linear_workspace_size(int32_t M, int32_t N,
                                              int32_t K, int32_t epilogue) {
  if (!gemm_shape_ok(M, N, K) ||
      (epilogue != kStoreBf16 && epilogue != kAddF32 && epilogue != kSwiglu))
    return 0;
  return gemm_plan(M, N, K, epilogue).part_bytes;
}

extern "C" int wedlm_linear(const uint16_t* x, const uint16_t* w, int32_t M,
                            int32_t N, int32_t K, int32_t epilogue, void* out,
                            int32_t ldo, void* workspace,
                            size_t workspace_bytes, void* stream) {
  return gemm(x, w, M, N, K, out, ldo, epilogue, workspace, workspace_bytes,
              false, false, static_cast<hipStream_t>(stream));
}

extern "C" int wedlm_qk_norm_rope(const uint16_t* qkv, const uint16_t* q_gain,
                                  const uint16_t* k_gain,
                                  const int32_t* pos_ids, int32_t M,
                                  int32_t Hq, int32_t Hkv, int32_t D,
                                  double rope_theta, float eps,
                                  uint16_t* q_out, uint16_t* k_out,
                                  uint16_t* v_out, void* stream) {
  if (!qkv || !q_gain || !k_gain || !pos_ids || !q_out || !k_out || !v_out)
    return WEDLM_E_ARG;
  if (!(rope_theta > 1.0) || !(eps > 0.f)) return WEDLM_E_ARG;
  if (M < 1 || Hq < 1 || Hkv < 1 || (D != 64 && D != 128)) return WEDLM_E_SHAPE;
  return qk_norm_rope(qkv, nullptr, 1, M, q_gain, k_gain, pos_ids, Hq, Hkv, D,
                      rope_theta, eps, q_out, k_out, v_out,
                      static_cast<hipStream_t>(stream));
}

extern "C" size_t wedlm_model_workspace_size(const wedlm_model_config* cfg,
                                             int32_t B, int32_t W,
                                             int32_t max_prefix_len) {
  if (!config_ok(cfg) || B < 1 || W < 1 || W > WEDLM_MAX_WINDOW ||
      max_prefix_len < 0)
    return 0;
  return carve(cfg, B, W, max_prefix_len).total;
}

extern "C" int wedlm_model_forward(
    const wedlm_model_config* cfg, const wedlm_model_weights* wt,
    const int32_t* win_tok, const int32_t* win_start, int32_t B, int32_t W,
    const uint16_t* k_cache, const uint16_t* v_cache, int64_t num_pages,
    const int32_t* block_table, int32_t max_pages, int32_t max_prefix_len,
    double temperature, int32_t* perm, int32_t* pos_ids, int32_t* tok_phys,
    int32_t* n_obs, uint16_t* k_win, uint16_t* v_win, int32_t* argmax,
    float* entropy, float* pmax, int32_t* status, void* workspace,
    size_t workspace_bytes, void* stream) {
  if (!cfg || !wt || !win_tok || !win_start || !k_cache || !v_cache ||
      !block_table || !perm || !pos_ids || !tok_phys || !n_obs || !k_win ||
      !v_win || !argmax || !entropy || !status)
    return WEDLM_E_ARG;
  if (!wt->embed || !wt->attn_norm || !wt->w_qkv || !wt->q_norm ||
      !wt->k_norm || !wt->w_o || !wt->mlp_norm || !wt->w_gate_up ||
      !wt->w_down || !wt->final_norm || !wt->lm_head)
    return WEDLM_E_ARG;
  if (!(temperature > 0.0)) return WEDLM_E_ARG;
  if (!config_ok(cfg) || B < 1 || W < 1 || W > WEDLM_MAX_WINDOW ||
      max_prefix_len < 0 || num_pages < 1)
    return WEDLM_E_SHAPE;
  const Carve cv = carve(cfg, B, W, max_prefix_len);
  if (!workspace || workspace_bytes < cv.total) return WEDLM_E_WORKSPACE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  float* x = reinterpret_cast<float*>(ws + cv.x);
  uint16_t* xn = reinterpret_cast<uint16_t*>(ws + cv.xn);
  uint16_t* qkv = reinterpret_cast<uint16_t*>(ws + cv.qkv);
  uint16_t* q = reinterpret_cast<uint16_t*>(ws + cv.q);
  uint16_t* attn = reinterpret_cast<uint16_t*>(ws + cv.attn);
  uint16_t* act = reinterpret_cast<uint16_t*>(ws + cv.act);
  float* part = reinterpret_cast<float*>(ws + cv.part);
  const size_t part_bytes = cv.part_bytes;
  void* attn_ws = ws + cv.attn_ws;
  void* lm_ws = ws + cv.lm_ws;
  const size_t attn_ws_bytes = cv.lm_ws - cv.attn_ws;
  const size_t lm_ws_bytes = cv.total - cv.lm_ws;

  const int M = B * W;
  const int Hd = cfg->hidden, Hq = cfg->n_heads, Hkv = cfg->n_kv_heads;
  const int D = cfg->head_dim, I = cfg->inter;
  const int QKV = (Hq + 2 * Hkv) * D;
  const int64_t win_stride = static_cast<int64_t>(M) * Hkv * D;
  const int64_t cache_stride = num_pages * Hkv * kPage * D;
  const float scale = 1.0f / sqrtf(static_cast<float>(D));
  int rc;
#define WEDLM_TRY(call) \
  if ((rc = (call)) != WEDLM_OK) return rc

  // physical order of the window (Eq. 5/6) and its positions (Eq. 2)
  WEDLM_TRY(wedlm_reorder(win_tok, win_start, nullptr, B, W, Hq, Hkv, D,
                          cfg->rope_theta, perm, pos_ids, tok_phys, n_obs,
                          nullptr, nullptr, nullptr, stream));
  WEDLM_TRY(wedlm_embed(tok_phys, M, cfg->mask_token, wt->embed, cfg->vocab,
                        Hd, x, stream));
  // pend > 1: split partials of the last residual-add product, summed into
  // x by the next RMSNorm
  int pend = 0;
  for (int l = 0; l < cfg->n_layers; ++l) {
    uint16_t* kl = k_win + l * win_stride;
    uint16_t* vl = v_win + l * win_stride;
    WEDLM_TRY(norm(x, part, pend, M, Hd,
                   wt->attn_norm + static_cast<int64_t>(l) * Hd, cfg->rms_eps,
                   xn, true, st));
    // a split q|k|v product leaves fp32 partials, summed by the q/k norm
    int qkv_ks = 1;
    WEDLM_TRY(gemm(xn, wt->w_qkv + static_cast<int64_t>(l) * QKV * Hd, M, QKV,
                   Hd, qkv, QKV, kStoreBf16, part, part_bytes, true, true, st,
                   &qkv_ks));
    WEDLM_TRY(qk_norm_rope(qkv, part, qkv_ks, M,
                           wt->q_norm + static_cast<int64_t>(l) * D,
                           wt->k_norm + static_cast<int64_t>(l) * D, pos_ids,
                           Hq, Hkv, D, cfg->rope_theta, cfg->rms_eps, q, kl,
                           vl, st));
    // the attention writes its output in the packed tile layout that the
    // output projection reads
    WEDLM_TRY(window_attn_packed(
        q, kl, vl, k_cache + l * cache_stride, v_cache + l * cache_stride,
        num_pages, block_table, max_pages, win_start, B, W, Hq, Hkv, D,
        max_prefix_len, scale, attn, status, attn_ws, attn_ws_bytes, stream));
    WEDLM_TRY(gemm(attn, wt->w_o + static_cast<int64_t>(l) * Hd * Hq * D, M,
                   Hd, Hq * D, x, Hd, kAddF32, part, part_bytes, true, true,
                   st, &pend));
    WEDLM_TRY(norm(x, part, pend, M, Hd,
                   wt->mlp_norm + static_cast<int64_t>(l) * Hd, cfg->rms_eps,
                   xn, true, st));
    WEDLM_TRY(gemm(xn, wt->w_gate_up + static_cast<int64_t>(l) * 2 * I * Hd, M,
                   I, Hd, act, I, kSwiglu, nullptr, 0, true, true, st));
    WEDLM_TRY(gemm(act, wt->w_down + static_cast<int64_t>(l) * Hd * I, M, Hd,
                   I, x, Hd, kAddF32, part, part_bytes, true, true, st,
                   &pend));
  }
  WEDLM_TRY(norm(x, part, pend, M, Hd, wt->final_norm, cfg->rms_eps, xn, false,
                 st));
  WEDLM_TRY(wedlm_lm_head_score(xn, wt->lm_head, M, Hd, cfg->vocab,
                                temperature, argmax, entropy, pmax, lm_ws,
                                lm_ws_bytes, stream));
#undef WEDLM_TRY
  return WEDLM_OK;
}
