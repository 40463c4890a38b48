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
// Accuracy of e^z: the exponent y = (l - m) * log2(e)/T (m the wave's
// running maximum) is formed in fp32 as fma(d, c2h, d * c2l) with
// d = l - m (exact when l and m are close) and log2(e)/T = c2h + c2l split
// into an fp32 head and tail, so no rounding is shared by all the terms of
// a row; v_exp_f32 gives 2^y.  Only the rescaling of a state to a new
// maximum evaluates its exponent in fp64.
//
// Roofline: 4*V bytes per masked row, read once.
// Work: with 512 rows or more, one workgroup per row (observed rows exit)
// and no partials.  With fewer rows the chunking follows the rows that are
// masked in this call, known only on the device: every workgroup counts
// them (Mt, from n_obs), splits each into nch = ceil(768 / Mt) vocabulary
// chunks of at least 16K logits, and takes item g = (masked row g / nch,
// chunk g % nch) of the compacted list, so about 768 workgroups stream
// whatever the share of observed rows; a merge kernel combines the chunks.
#include <algorithm>

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
  int B, W, V;
  int dyn;                     // chunks from the masked rows (fewer than 1024 rows)
  int max_nchunk;              // dyn: chunks per row at most (>= 8K logits each)
  double c2;
  int32_t* argmax;
  float* entropy;
  float* pmax;
  State* ws;                   // dyn: [B*W, max_nchunk] partials by masked row
};

// About three workgroups per CU, chunks of at least 16K logits: 1152
// workgroups at 384 masked rows and 8K chunks at 16 rows measured 9% and
// 7% slower.
constexpr int kTargetWgs = 768;
constexpr int kMinChunk = 16384;          // logits per chunk at least

__device__ __forceinline__ int clamp_obs(const ScoreArgs& a, int b) {
  const int no = a.n_obs[b];
  return no < 0 ? 0 : (no > a.W ? a.W : no);
}

// The masked rows of the call: sequences in order, rows in order within a
// sequence.  The first 64 sequences' counts and their inclusive prefix sums
// are kept in registers (one lane each), so with up to 64 sequences n_obs
// is read once; further groups of 64 are re-read on demand.
struct MaskedRows {
  int no0, c0, inc0;   // this lane's sequence of the first group
  int total;           // masked rows over all sequences (wave-uniform)
};

__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int t = __shfl_up(v, off);
    if (lane >= off) v += t;
  }
  return v;
}

__device__ MaskedRows masked_rows(const ScoreArgs& a) {
  MaskedRows m;
  const int lane = lane_id();
  m.no0 = lane < a.B ? clamp_obs(a, lane) : a.W;
  m.c0 = a.W - m.no0;
  m.inc0 = wave_incl_scan(m.c0);
  m.total = __shfl(m.inc0, kWave - 1);
  for (int b0 = kWave; b0 < a.B; b0 += kWave) {
    const int b = b0 + lane;
    int c = b < a.B ? a.W - clamp_obs(a, b) : 0;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) c += __shfl_xor(c, off);
    m.total += c;
  }
  return m;
}

// The r-th masked row (0 <= r < total; r wave-uniform) as (b, i).
__device__ void masked_row(const ScoreArgs& a, const MaskedRows& m, int r,
                           int& b_out, int& i_out) {
  int base = 0, no = m.no0, c = m.c0, inc = m.inc0;
  for (int b0 = 0; b0 < a.B; b0 += kWave) {
    if (b0 > 0) {
      const int b = b0 + lane_id();
      no = b < a.B ? clamp_obs(a, b) : a.W;
      c = a.W - no;
      inc = wave_incl_scan(c);
    }
    const int tot = __shfl(inc, kWave - 1);
    if (r < base + tot) {
      const uint64_t hit = ballot(base + inc > r);
      const int L = __ffsll(static_cast<unsigned long long>(hit)) - 1;
      const int excl = __shfl(inc - c, L);
      b_out = b0 + L;
      i_out = __shfl(no, L) + (r - base - excl);
      return;
    }
    base += tot;
  }
  b_out = 0;
  i_out = 0;
}

// Chunks per masked row and their length, from the masked-row count.
struct ChunkPlan {
  int nch, chunk;
};
__device__ __forceinline__ ChunkPlan chunk_plan(const ScoreArgs& a, int mt) {
  int n = (kTargetWgs + mt - 1) / mt;
  n = n > a.max_nchunk ? a.max_nchunk : n;
  n = n < 1 ? 1 : n;
  ChunkPlan p;
  p.chunk = (((a.V + n - 1) / n) + 3) & ~3;
  p.nch = (a.V + p.chunk - 1) / p.chunk;
  return p;
}

// kVec: rows start on 16-byte boundaries (row_stride % 4 == 0 and an
// aligned base), so the body streams 16-byte loads; otherwise 4-byte loads.
// Thread t takes float4 groups t, t+256, ... of the chunk, four at a time.
template <bool kVec>
__global__ __launch_bounds__(kThreads) void score_kernel(ScoreArgs a) {
  int row, ch = 0, v0 = 0, v1 = a.V, r = 0, nch = 1;
  if (a.dyn) {
    const MaskedRows mr = masked_rows(a);
    const ChunkPlan cp = chunk_plan(a, mr.total);
    nch = cp.nch;
    if (static_cast<int>(blockIdx.x) >= mr.total * nch) return;
    r = blockIdx.x / nch;
    ch = blockIdx.x - r * nch;
    int b, i;
    masked_row(a, mr, r, b, i);
    row = b * a.W + i;
    v0 = ch * cp.chunk;
    v1 = min(a.V, v0 + cp.chunk);
  } else {
    row = blockIdx.x;
    const int b = row / a.W;
    if (row - b * a.W < clamp_obs(a, b)) return;
  }
  const float* x = a.logits + static_cast<int64_t>(row) * a.row_stride;
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
  if (!a.dyn) finish(st, row, a.argmax, a.entropy, a.pmax);
  else a.ws[static_cast<int64_t>(r) * a.max_nchunk + ch] = st;
}

// Merge the chunk partials of each masked row, in chunk order (dyn only;
// workgroup g takes masked row g).
__global__ __launch_bounds__(kWave) void score_merge_kernel(ScoreArgs a) {
  const MaskedRows mr = masked_rows(a);
  const int r = blockIdx.x;
  if (r >= mr.total) return;
  const int nch = chunk_plan(a, mr.total).nch;
  int b, i;
  masked_row(a, mr, r, b, i);
  State st = empty_state();
  const State* p = a.ws + static_cast<int64_t>(r) * a.max_nchunk;
  for (int c = lane_id(); c < nch; c += kWave) merge(st, p[c], a.c2);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) merge(st, shfl_xor_state(st, off), a.c2);
  if (lane_id() == 0) finish(st, b * a.W + i, a.argmax, a.entropy, a.pmax);
}

// Window rows from which every row takes one workgroup, unchunked: at 512
// rows (384 masked at long_prefix, about 222 in the streaming loop) the
// merge kernel's launch cost more than the chunks gained (score 45.5
// against 48.8 us at long_prefix, the loop's step 0.137 against 0.138 ms).
constexpr int kWholeRows = 512;

// Chunks per row at most (0: no chunking, one workgroup per row): with
// fewer than kWholeRows rows and a vocabulary of more than one 16K chunk.
int plan_max_nchunk(int B, int W, int V) {
  if (static_cast<int64_t>(B) * W >= kWholeRows) return 0;
  const int n = (V + kMinChunk - 1) / kMinChunk;
  return n > 1 ? n : 0;
}

}  // namespace

extern "C" size_t wedlm_score_workspace_size(int32_t B, int32_t W, int32_t V) {
  if (B < 1 || W < 1 || W > WEDLM_MAX_WINDOW || V < 1) return 0;
  const int mx = plan_max_nchunk(B, W, V);
  return mx > 0 ? static_cast<size_t>(B) * W * mx * sizeof(State) : 0;
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
  a.max_nchunk = plan_max_nchunk(B, W, V);
  a.dyn = a.max_nchunk > 0;
  a.c2 = 1.4426950408889634074 / temperature;
  a.argmax = argmax; a.entropy = entropy; a.pmax = pmax;
  const size_t need = wedlm_score_workspace_size(B, W, V);
  if (workspace_bytes < need || (need && !workspace)) return WEDLM_E_WORKSPACE;
  a.ws = static_cast<State*>(workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const bool vec = (row_stride & 3) == 0 &&
                   (reinterpret_cast<uintptr_t>(logits) & 15) == 0;
  // dyn: at most masked rows x ceil(768 / masked rows) items, i.e. fewer
  // than 768 + B*W, and at most B*W x max_nchunk
  const int rows = B * W;
  const int grid = a.dyn ? std::min(kTargetWgs + rows, rows * a.max_nchunk) : rows;
  if (vec)
    hipLaunchKernelGGL(score_kernel<true>, dim3(grid), dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL(score_kernel<false>, dim3(grid), dim3(kThreads), 0, st, a);
  WEDLM_LAUNCH_CHECK();
  if (a.dyn) {
    hipLaunchKernelGGL(score_merge_kernel, dim3(B * W), dim3(kWave), 0, st, a);
    WEDLM_LAUNCH_CHECK();
  }
  return WEDLM_OK;
}
