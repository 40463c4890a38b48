// Greedy token and entropy of every mask slot's predicted distribution
// (Sec. 5.2, the H_i of Eq. (11)).
//
// One pass over each masked row's fp32 logits.  Every thread keeps an online
// state (max logit l_max, its lowest index, R = sum_{v != argmax} e^{z_v},
// S = sum_{v != argmax} -z_v e^{z_v}, z_v = (l_v - l_max)/T) with R and S in
// fp64; states merge associatively across lanes, waves and vocabulary
// chunks, ties going to the lower token id.  Then
//   H = ln(1 + R) + S / (1 + R),   p_max = 1 / (1 + R),
// two non-negative terms, so nothing cancels even when H is ~1e-25 (strongly
// peaked rows at T = 0.1).
//
// Accuracy of e^z: the exponent y = (l - l_max) * log2(e)/T is formed in
// fp64, split into y_hi = fp32(y) and y_lo = y - y_hi, and
// 2^y = v_exp_f32(y_hi) * (1 + y_lo ln 2), which keeps the relative error of
// each term near one fp32 ulp even at |y| ~ 150.
//
// Roofline: 4*V bytes per masked row, read once; grid = masked rows x
// vocabulary chunks, chunks sized so that every CU has work.
#include "common.h"
#include "score_state.h"

using namespace wedlm;

namespace {

constexpr int kThreads = 256;
constexpr int kBlk = 16;                 // logits per thread per step

// Reduce the block's states into thread 0's.
__device__ State block_reduce(State st, double c2) {
  __shared__ State sh[kThreads / kWave];
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) merge(st, shfl_xor_state(st, off), c2);
  const int wave = threadIdx.x / kWave;
  if (lane_id() == 0) sh[wave] = st;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kThreads / kWave; ++w) merge(st, sh[w], c2);
  }
  return st;
}

struct ScoreArgs {
  const float* logits;
  int64_t row_stride;
  const int32_t* n_obs;
  int B, W, V, nchunk, chunk;  // chunk: elements per chunk (multiple of 4)
  double c2;
  int32_t* argmax;
  float* entropy;
  float* pmax;
  State* ws;                   // [B*W, nchunk] partials (nchunk > 1)
};

// kVec: rows start on 16-byte boundaries (row_stride % 4 == 0 and an
// aligned base), so the body streams 16-byte loads; otherwise 4-byte loads.
// Thread t takes float4 groups t, t+256, ... of the chunk, four at a time.
template <bool kVec>
__global__ __launch_bounds__(kThreads) void score_kernel(ScoreArgs a) {
  const int ch = blockIdx.x % a.nchunk;
  const int row = blockIdx.x / a.nchunk;
  const int b = row / a.W;
  const int i = row - b * a.W;
  int no = a.n_obs[b];
  no = no < 0 ? 0 : (no > a.W ? a.W : no);
  if (i < no) return;
  const float* x = a.logits + static_cast<int64_t>(row) * a.row_stride;
  const int v0 = ch * a.chunk;
  const int v1 = min(a.V, v0 + a.chunk);
  State st = empty_state();
  const ExpScale sc = exp_scale(a.c2);
  constexpr int kStep = kThreads * kBlk;       // logits per workgroup step
  int v = v0;
  if (kVec) {
    // full steps, loads one step ahead of the arithmetic (the prefetch of
    // the last step re-reads it, so every load is unconditional and in
    // bounds and the wait before each step leaves the next one in flight)
    const int nsteps = (v1 - v0) / kStep;
    auto load = [&](int s, floatx4_t (&q)[kBlk / 4]) {
      const int vs = v0 + s * kStep;
#pragma unroll
      for (int g = 0; g < kBlk / 4; ++g)
        q[g] = __builtin_nontemporal_load(reinterpret_cast<const floatx4_t*>(
            x + vs + (g * kThreads + threadIdx.x) * 4));
    };
    auto consume = [&](int s, const floatx4_t (&q)[kBlk / 4]) {
      const int vs = v0 + s * kStep;
      float xs[kBlk];
      int idx[kBlk];
#pragma unroll
      for (int g = 0; g < kBlk / 4; ++g)
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          xs[g * 4 + k] = q[g][k];
          idx[g * 4 + k] = vs + (g * kThreads + threadIdx.x) * 4 + k;
        }
      push_block(st, xs, idx, sc);
    };
    if (nsteps > 0) {
      floatx4_t qa[kBlk / 4], qb[kBlk / 4];
      load(0, qa);
      int s = 0;
      for (; s + 2 <= nsteps; s += 2) {
        load(min(s + 1, nsteps - 1), qb);
        consume(s, qa);
        load(min(s + 2, nsteps - 1), qa);
        consume(s + 1, qb);
      }
      if (s < nsteps) consume(s, qa);
    }
    v = v0 + nsteps * kStep;
  }
  // remainder (and the whole chunk without 16-byte alignment): one logit at
  // a time in increasing index order per thread
  for (int u = v + threadIdx.x; u < v1; u += kThreads) {
    const float xs[1] = {x[u]};
    const int idx[1] = {u};
    push_block(st, xs, idx, sc);
  }
  st = block_reduce(st, a.c2);
  if (threadIdx.x != 0) return;
  if (a.nchunk == 1) finish(st, row, a.argmax, a.entropy, a.pmax);
  else a.ws[static_cast<int64_t>(row) * a.nchunk + ch] = st;
}

// Merge the chunk partials of each masked row, in chunk order.
__global__ __launch_bounds__(kWave) void score_merge_kernel(ScoreArgs a) {
  const int row = blockIdx.x;
  const int b = row / a.W;
  const int i = row - b * a.W;
  int no = a.n_obs[b];
  no = no < 0 ? 0 : (no > a.W ? a.W : no);
  if (i < no) return;
  State st = empty_state();
  const State* p = a.ws + static_cast<int64_t>(row) * a.nchunk;
  for (int c = lane_id(); c < a.nchunk; c += kWave) merge(st, p[c], a.c2);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) merge(st, shfl_xor_state(st, off), a.c2);
  if (lane_id() == 0) finish(st, row, a.argmax, a.entropy, a.pmax);
}

int plan_chunks(int B, int W, int V, int* chunk) {
  // about 768 workgroups over the B*W rows and at least two chunks per
  // row, each chunk >= 16K elements: long enough that the per-workgroup
  // merge is a small share, short enough that loads stay in flight
  const int rows = B * W;
  int nchunk = (768 + rows - 1) / rows;
  if (nchunk < 2) nchunk = 2;
  const int max_by_size = (V + 16383) / 16384;
  if (nchunk > max_by_size) nchunk = max_by_size;
  if (nchunk < 1) nchunk = 1;
  int c = (V + nchunk - 1) / nchunk;
  c = (c + 3) & ~3;
  nchunk = (V + c - 1) / c;
  *chunk = c;
  return nchunk;
}

}  // namespace

extern "C" size_t wedlm_score_workspace_size(int32_t B, int32_t W, int32_t V) {
  if (B < 1 || W < 1 || W > WEDLM_MAX_WINDOW || V < 1) return 0;
  int chunk;
  const int nchunk = plan_chunks(B, W, V, &chunk);
  return nchunk > 1 ? static_cast<size_t>(B) * W * nchunk * sizeof(State) : 0;
}

extern "C" int wedlm_score(const float* logits, int64_t row_stride,
                           const int32_t* n_obs, int32_t B, int32_t W,
                           int32_t V, double temperature, int32_t* argmax,
                           float* entropy, float* pmax, void* workspace,
                           size_t workspace_bytes, void* stream) {
  if (!logits || !n_obs || !argmax || !entropy) return WEDLM_E_ARG;
  if (!(temperature > 0.0) || !(temperature < 1e30)) return WEDLM_E_ARG;
  if (B < 1 || W < 1 || W > WEDLM_MAX_WINDOW || V < 1 || row_stride < V ||
      static_cast<int64_t>(B) * W > (1ll << 24))
    return WEDLM_E_SHAPE;
  ScoreArgs a{};
  a.logits = logits; a.row_stride = row_stride; a.n_obs = n_obs;
  a.B = B; a.W = W; a.V = V;
  a.nchunk = plan_chunks(B, W, V, &a.chunk);
  a.c2 = 1.4426950408889634074 / temperature;
  a.argmax = argmax; a.entropy = entropy; a.pmax = pmax;
  const size_t need = wedlm_score_workspace_size(B, W, V);
  if (workspace_bytes < need || (need && !workspace)) return WEDLM_E_WORKSPACE;
  a.ws = static_cast<State*>(workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool vec = (row_stride & 3) == 0 &&
                   (reinterpret_cast<uintptr_t>(logits) & 15) == 0;
  if (vec)
    hipLaunchKernelGGL(score_kernel<true>, dim3(B * W * a.nchunk),
                       dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL(score_kernel<false>, dim3(B * W * a.nchunk),
                       dim3(kThreads), 0, st, a);
  WEDLM_LAUNCH_CHECK();
  if (a.nchunk > 1) {
    hipLaunchKernelGGL(score_merge_kernel, dim3(B * W), dim3(kWave), 0, st, a);
    WEDLM_LAUNCH_CHECK();
  }
  return WEDLM_OK;
}
