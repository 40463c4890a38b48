// Greedy token and entropy of every mask slot's predicted distribution
// (Sec. 5.2, the H_i of Eq. (11)).
//
// One pass over each masked row's fp32 logits.  Every thread keeps an online
// state (max logit l_max, its lowest index, exact tie count,
// R = sum_{v != argmax} e^{z_v}, S = sum_{v != argmax} -z_v e^{z_v},
// z_v = (l_v - l_max)/T) with R and S accumulated per block in fp32 and
// carried in fp64; states merge associatively across lanes, waves and
// vocabulary chunks, ties going to the lower token id.  Then
//   H = ln(1 + R) + S / (1 + R),   p_max = 1 / (1 + R),
// two non-negative terms, so nothing cancels even when H is ~1e-25 (strongly
// peaked rows at T = 0.1).
//
// Accuracy of e^z (score_state.h): the exponent y = (l - l_max) * log2(e)/T
// is formed in fp32 from split constants, log2(e)/T = c2h + c2l and
// l_max * c2h = mch + mcl (its exact fused-multiply-add residual), as
// fma(l, c2h, -mch) - mcl + (l - l_max) * c2l; no rounding is shared by all
// the terms of a row, and v_exp_f32 gives 2^y.  Only the rescaling of a
// state to a new maximum evaluates its exponent in fp64.
//
// Roofline: 4*V bytes per masked row, read once; grid = masked rows x
// vocabulary chunks, chunks sized so that every CU has work.
#include "common.h"
#include "score_state.h"

using namespace wedlm;

namespace {

constexpr int kThreads = 256;
constexpr int kBlk = 8;                  // logits per thread per step

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

// Maximum of v over the wave's 64 lanes (every lane gets it).
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

// Three-input maximum of finite or -inf values (v_max3_f32).
__device__ __forceinline__ float max3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Add a block of N logits per lane (indices idx, increasing within a lane)
// to the lane's state, where every lane of the wave keeps the same running
// maximum st.m (the wave's).  A raise is then wave-uniform and rare: only
// when some lane's block beats everything the wave has seen.  When no
// lane's block reaches st.m (every step but those few), every term is added
// with no tie handling; otherwise every lane counts its exact ties with
// st.m and the lowest index among them.
template <int N>
__device__ __forceinline__ void push_block_wave(State& st,
                                                const float (&x)[N],
                                                const int (&idx)[N],
                                                const ExpScale& sc) {
  static_assert(N % 2 == 0, "pairs of logits per v_max3");
  float bm = x[0];
#pragma unroll
  for (int k = 1; k < N; k += 2) bm = max3(bm, x[k], x[k + 1 < N ? k + 1 : k]);
  if (ballot(bm > st.m)) {
    const float wm = wave_max(bm);
    shift_state(st, wm, sc.c2);
    st.m = wm;
    st.tok = 0x7fffffff;
  }
  // y = (x - m) * c2 as d*c2h + d*c2l with d = x - m: no rounding shared by
  // the terms of a row; clamped at -256 (a -inf logit, or the NaN of an
  // empty state, adds 0, never inf * 0)
  const float m = st.m;
  float r = 0.f, sy = 0.f;
  if (ballot(bm == m)) {
    int ties = 0;
#pragma unroll
    for (int k = 0; k < N; ++k) {
      const float d = x[k] - m;
      const float y =
          fmaxf(__builtin_fmaf(d, sc.c2h, d * sc.c2l), -256.f);
      const bool is_max = x[k] == m;
      const float e = is_max ? 0.f : __builtin_amdgcn_exp2f(y);
      ties += is_max ? 1 : 0;
      r += e;
      sy = __builtin_fmaf(-y, e, sy);
    }
    if (ties) {
      int t = 0x7fffffff;
#pragma unroll
      for (int k = N - 1; k >= 0; --k) t = x[k] == m ? idx[k] : t;
      st.ties += ties;
      st.tok = min(st.tok, t);
    }
  } else {
#pragma unroll
    for (int k = 0; k < N; ++k) {
      const float d = x[k] - m;
      const float y =
          fmaxf(__builtin_fmaf(d, sc.c2h, d * sc.c2l), -256.f);
      const float e = __builtin_amdgcn_exp2f(y);
      r += e;
      sy = __builtin_fmaf(-y, e, sy);
    }
  }
  st.R += r;
  st.S += sy;
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
    // full steps, loads two steps ahead of the arithmetic (the prefetches
    // past the last step re-read it, so every load is unconditional and in
    // bounds and the wait before each step leaves the next two in flight)
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
      push_block_wave(st, xs, idx, sc);
    };
    if (nsteps > 0) {
      floatx4_t qa[kBlk / 4], qb[kBlk / 4], qc[kBlk / 4];
      load(0, qa);
      load(min(1, nsteps - 1), qb);
      int s = 0;
      for (; s + 3 <= nsteps; s += 3) {
        load(min(s + 2, nsteps - 1), qc);
        consume(s, qa);
        load(min(s + 3, nsteps - 1), qa);
        consume(s + 1, qb);
        load(min(s + 4, nsteps - 1), qb);
        consume(s + 2, qc);
      }
      if (s < nsteps) consume(s, qa);
      if (s + 1 < nsteps) consume(s + 1, qb);
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
  // about 1024 workgroups over the B*W rows (four per CU), each chunk >= 16K
  // elements: long enough that the per-workgroup merge is a small share,
  // short enough that loads stay in flight.  With 1024 rows or more, one
  // chunk per row: no partials and no merge kernel.
  const int rows = B * W;
  int nchunk = (1024 + rows - 1) / rows;
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
