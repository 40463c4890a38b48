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

using namespace wedlm;

namespace {

constexpr int kThreads = 256;
constexpr double kLn2 = 0.69314718055994530942;

struct State {
  float m;      // max logit
  int tok;      // its lowest index
  double R;     // sum over v != tok of 2^{y_v}
  double S;     // sum over v != tok of -y_v 2^{y_v}  (log2 units)
};

__device__ __forceinline__ State empty_state() {
  return State{kNegInf, 0x7fffffff, 0.0, 0.0};
}

// 2^y for y <= 0 (fp64 argument), relative error ~1 fp32 ulp; 0 below -200.
__device__ __forceinline__ double exp2_acc(double y) {
  if (!(y > -200.0)) return 0.0;
  const float yh = static_cast<float>(y);
  const double yl = y - static_cast<double>(yh);
  const double e = static_cast<double>(__builtin_amdgcn_exp2f(yh));
  return __fma_rn(e, yl * kLn2, e);
}

// Add one element (value x at index v) to a state.  c2 = log2(e) / T.
__device__ __forceinline__ void push(State& st, float x, int v, double c2) {
  if (x > st.m) {
    if (st.m != kNegInf) {
      // the old maximum joins the sums; every old term shifts by dy < 0
      const double dy = (static_cast<double>(st.m) - x) * c2;
      const double e = exp2_acc(dy);
      st.S = e * (st.S - dy * (st.R + 1.0));
      st.R = e * (st.R + 1.0);
      if (e == 0.0) st.S = 0.0;
    }
    st.m = x;
    st.tok = v;
  } else {
    const double y = (static_cast<double>(x) - st.m) * c2;
    const double e = exp2_acc(y);
    st.R += e;
    if (e > 0.0) st.S = __fma_rn(-y, e, st.S);
  }
}

// Merge state o into st.  The winner keeps its maximum; the loser's terms,
// its own maximum included, shift by dy = (m_loser - m_winner) * c2 <= 0.
__device__ __forceinline__ void merge(State& st, const State& o, double c2) {
  if (o.m == kNegInf) return;
  if (st.m == kNegInf) { st = o; return; }
  const bool keep = (st.m > o.m) || (st.m == o.m && st.tok < o.tok);
  const State& w = keep ? st : o;
  const State& l = keep ? o : st;
  const double dy = (static_cast<double>(l.m) - w.m) * c2;
  const double e = exp2_acc(dy);
  double R = w.R + e * (l.R + 1.0);
  double S = w.S;
  if (e > 0.0) S += e * (l.S - dy * (l.R + 1.0));
  st = State{w.m, w.tok, R, S};
}

__device__ __forceinline__ State shfl_xor_state(const State& s, int mask) {
  State o;
  o.m = __shfl_xor(s.m, mask);
  o.tok = __shfl_xor(s.tok, mask);
  o.R = __shfl_xor(s.R, mask);
  o.S = __shfl_xor(s.S, mask);
  return o;
}

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

__device__ __forceinline__ void finish(const State& st, int64_t idx,
                                       int32_t* argmax, float* entropy,
                                       float* pmax) {
  const double S = st.S * kLn2;            // back to nats
  const double H = log1p(st.R) + S / (1.0 + st.R);
  argmax[idx] = st.m == kNegInf ? 0 : st.tok;   // an all -inf row: id 0
  entropy[idx] = static_cast<float>(H);
  if (pmax) pmax[idx] = static_cast<float>(1.0 / (1.0 + st.R));
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
  // chunk bounds are multiples of 4 elements, the row tail may not be
  const int v1v = kVec ? v0 + ((v1 - v0) & ~3) : v0;
  if (kVec) {
    for (int v = v0 + threadIdx.x * 4; v < v1v; v += kThreads * 4) {
      const floatx4_t q = *reinterpret_cast<const floatx4_t*>(x + v);
      push(st, q[0], v, a.c2);
      push(st, q[1], v + 1, a.c2);
      push(st, q[2], v + 2, a.c2);
      push(st, q[3], v + 3, a.c2);
    }
  }
  for (int v = v1v + threadIdx.x; v < v1; v += kThreads) push(st, x[v], v, a.c2);
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
  // aim for >= 2048 workgroups over the B*W rows, chunks >= 16K elements
  const int rows = B * W;
  int nchunk = (2048 + rows - 1) / rows;
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
