// Topological reordering (Eq. 5/6) and RoPE at logical positions (Eq. 2).
//
// One workgroup per (physical row i, sequence b).  Wave 0 rebuilds the
// stable partition of the window from two ballots: physical row i < n_obs
// takes the i-th filled slot, row i >= n_obs the (i - n_obs)-th mask slot.
// The row's angles are computed once in fp64 and shared through LDS; every
// query and key head of the row is rotated in fp64 and rounded to bf16 (16
// bytes per load and store), the value heads are copied.  The kernel moves
// (Hq + 2 Hkv) * D * 2 bytes in and out per row; it is small next to
// attention and scoring, and bound by the latency of its round trips.
#include "common.h"

using namespace wedlm;

namespace {

constexpr int kThreads = 256;
constexpr int kMaxHalf = 64;   // D/2 for D <= 128

__global__ __launch_bounds__(kThreads) void reorder_rope_kernel(
    const int32_t* __restrict__ win_tok, const int32_t* __restrict__ win_start,
    const uint16_t* __restrict__ qkv_in, int W, int Hq, int Hkv, int D,
    double theta, int32_t* __restrict__ perm, int32_t* __restrict__ pos_ids,
    int32_t* __restrict__ tok_phys, int32_t* __restrict__ n_obs,
    uint16_t* __restrict__ q_phys, uint16_t* __restrict__ k_phys,
    uint16_t* __restrict__ v_phys) {
  const int i = blockIdx.x;
  const int b = blockIdx.y;
  __shared__ int s_src;
  __shared__ double s_cos[kMaxHalf], s_sin[kMaxHalf];

  if (threadIdx.x < kWave) {
    const int s = threadIdx.x;
    const int t = (s < W) ? win_tok[b * W + s] : 0;
    const uint64_t filled = ballot(s < W && t >= 0);
    const uint64_t masked = ballot(s < W && t < 0);
    const int n_o = __popcll(filled);
    const uint64_t bits = (i < n_o) ? filled : masked;
    const int k = (i < n_o) ? i : i - n_o;
    const uint64_t below = (s == 0) ? 0ull : (bits & (~0ull >> (64 - s)));
    const bool hit = ((bits >> s) & 1ull) && __popcll(below) == k;
    const int src = __ffsll(static_cast<long long>(ballot(hit))) - 1;
    const int tok_src = __shfl(t, src);
    if (s == 0) {
      const int c = win_start[b];
      s_src = src;
      perm[b * W + i] = src;
      pos_ids[b * W + i] = c + src;
      tok_phys[b * W + i] = tok_src < 0 ? WEDLM_MASK_TOKEN : tok_src;
      if (i == 0) n_obs[b] = n_o;
    }
  }
  __syncthreads();
  if (qkv_in == nullptr) return;                  // indices only (uniform)
  const int src = s_src;
  const int half = D / 2;
  const int H = Hq + 2 * Hkv;
  const uint16_t* x = qkv_in + (static_cast<int64_t>(b) * W + src) * H * D;
  // one item = 8 consecutive rotation pairs of one query or key head (two
  // 16-byte loads, two 16-byte stores).  The first two rounds of items and
  // the first round of the value copy are loaded before the angles are
  // computed, so that one round trip covers a row of up to 512 items (the
  // fp64 pow and sincos run under it)
  const int chunks = half / 8;                     // items per head
  const int n_items = (Hq + Hkv) * chunks;
  const int nv = Hkv * D / 8;                      // 16-byte pieces of v
  auto load_item = [&](int it, u16x8_t& lo8, u16x8_t& hi8) {
    if (it < n_items) {
      const int head = it / chunks, j0 = (it - head * chunks) * 8;
      lo8 = *reinterpret_cast<const u16x8_t*>(x + head * D + j0);
      hi8 = *reinterpret_cast<const u16x8_t*>(x + head * D + j0 + half);
    }
  };
  const u16x8_t* xv = reinterpret_cast<const u16x8_t*>(x + (Hq + Hkv) * D);
  u16x8_t lo0 = {}, hi0 = {}, lo1 = {}, hi1 = {}, v0 = {};
  load_item(threadIdx.x, lo0, hi0);
  load_item(threadIdx.x + kThreads, lo1, hi1);
  if (static_cast<int>(threadIdx.x) < nv) v0 = xv[threadIdx.x];
  if (threadIdx.x < half) {
    const int j = threadIdx.x;
    const double pos = static_cast<double>(win_start[b]) + src;
    const double omega = pow(theta, -2.0 * j / D);
    double sn, cs;
    sincos(pos * omega, &sn, &cs);
    s_cos[j] = cs;
    s_sin[j] = sn;
  }
  __syncthreads();
  auto rotate = [&](int it, const u16x8_t& lo8, const u16x8_t& hi8) {
    if (it >= n_items) return;
    const int head = it / chunks, j0 = (it - head * chunks) * 8;
    u16x8_t olo, ohi;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const double a = bf16_to_f32(lo8[e]);
      const double c2 = bf16_to_f32(hi8[e]);
      const double cs = s_cos[j0 + e], sn = s_sin[j0 + e];
      olo[e] = f32_to_bf16(static_cast<float>(a * cs - c2 * sn));
      ohi[e] = f32_to_bf16(static_cast<float>(c2 * cs + a * sn));
    }
    uint16_t* dst =
        (head < Hq)
            ? q_phys + ((static_cast<int64_t>(b) * W + i) * Hq + head) * D
            : k_phys +
                  ((static_cast<int64_t>(b) * W + i) * Hkv + (head - Hq)) * D;
    *reinterpret_cast<u16x8_t*>(dst + j0) = olo;
    *reinterpret_cast<u16x8_t*>(dst + j0 + half) = ohi;
  };
  rotate(threadIdx.x, lo0, hi0);
  rotate(threadIdx.x + kThreads, lo1, hi1);
  for (int it = threadIdx.x + 2 * kThreads; it < n_items; it += kThreads) {
    u16x8_t lo8 = {}, hi8 = {};
    load_item(it, lo8, hi8);
    rotate(it, lo8, hi8);
  }
  // the value heads, 16 bytes per thread
  u16x8_t* dv = reinterpret_cast<u16x8_t*>(
      v_phys + (static_cast<int64_t>(b) * W + i) * Hkv * D);
  if (static_cast<int>(threadIdx.x) < nv) dv[threadIdx.x] = v0;
  for (int e = threadIdx.x + kThreads; e < nv; e += kThreads) dv[e] = xv[e];
}

}  // namespace

extern "C" int wedlm_reorder(const int32_t* win_tok, const int32_t* win_start,
                             const uint16_t* qkv_in, int32_t B, int32_t W,
                             int32_t Hq, int32_t Hkv, int32_t D,
                             double rope_theta, int32_t* perm,
                             int32_t* pos_ids, int32_t* tok_phys,
                             int32_t* n_obs, uint16_t* q_phys,
                             uint16_t* k_phys, uint16_t* v_phys,
                             void* stream) {
  if (!win_tok || !win_start || !perm || !pos_ids || !tok_phys || !n_obs)
    return WEDLM_E_ARG;
  // the gather and rotation are all or nothing: without them the call
  // computes the indices only
  const int given = !!qkv_in + !!q_phys + !!k_phys + !!v_phys;
  if (given != 0 && given != 4) return WEDLM_E_ARG;
  if (!(rope_theta > 1.0) || !(rope_theta < 1e300)) return WEDLM_E_ARG;
  if (B < 1 || B > 65535 || W < 1 || W > WEDLM_MAX_WINDOW || Hkv < 1 ||
      Hq < Hkv || Hq % Hkv != 0 || (D != 64 && D != 128) ||
      Hq + 2 * Hkv > 1024)
    return WEDLM_E_SHAPE;
  hipLaunchKernelGGL(reorder_rope_kernel, dim3(W, B), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), win_tok, win_start,
                     qkv_in, W, Hq, Hkv, D, rope_theta, perm, pos_ids,
                     tok_phys, n_obs, q_phys, k_phys, v_phys);
  WEDLM_LAUNCH_CHECK();
  return WEDLM_OK;
}
