// LM head fused with the score of each row: logits = hidden . W_vocab^T on
// bf16 MFMA, reduced on the fly to the greedy token, entropy and top
// probability of softmax(logits / T) (Sec. 5.2; the Forward of Algorithm 1
// produces the logits the mask slots are scored on).  The fp32 logits are
// never written to memory.
//
// Work decomposition:
//   workgroup = (256-row vocabulary tile, group of 32*NB hidden rows); eight
//               waves, wave w owns vocabulary rows 32w .. 32w+31 of the tile
//   MFMA      = v_mfma_f32_32x32x16_bf16 computing logits^T: A = 32 weight
//               rows x 16 k (registers), B = 16 k x 32 hidden rows (LDS)
//   k order   = the contraction runs over k in a permuted order that is the
//               same for A and B: in each 64-wide k step, lane half hf of
//               MFMA j takes k = 32*hf + 8*j .. +8.  Each lane's A operand
//               for a whole step is then 64 contiguous bytes of its weight
//               row (four 16-byte loads), the B operand 16 contiguous bytes
//               of an LDS row.
// Memory path: the weights are the HBM stream (V * Hd * 2 bytes per launch,
//   read once per row group); each wave streams its own rows straight into
//   registers, PF steps ahead.  The hidden rows of a step go through LDS
//   (XOR-swizzled 16-byte chunks), double-buffered, one barrier per step.
// Epilogue: a lane holds 16 logits of one hidden row per row block; they
//   enter the online score state of score_state.h, states merge across the
//   two lane halves, the eight waves (LDS) and the vocabulary tiles (a merge
//   kernel over a workspace of per-tile states).
// Roofline: 2 * R * Hd * V flops against V * Hd * 2 weight bytes per row
//   group; R rows in one group give an intensity of R flop/byte.
#include "common.h"
#include "score_state.h"

using namespace wedlm;

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * kWave;
constexpr int kVocabTile = 32 * kWaves;   // vocabulary rows per workgroup
constexpr int kKStep = 64;                // k per pipeline step
constexpr int kPF = 4;                    // weight steps in flight per wave

struct LmArgs {
  const uint16_t* hidden;   // [R, Hd]
  const uint16_t* w;        // [V, Hd]
  int R, Hd, V;
  int n_vt, n_rg;           // vocabulary tiles, row groups
  double c2;                // log2(e) / T
  int32_t* argmax;
  float* entropy;
  float* pmax;
  State* ws;                // [R, n_vt] (n_vt > 1)
};

// LDS row of one k step: 64 bf16 = eight 16-byte chunks; chunk c of row r
// sits in slot c ^ (r & 7), so the 8 lanes of one ds_read_b128 pass (8 rows,
// same chunk) hit 8 different slots.
__device__ __forceinline__ int h_off(int r, int c) {
  return r * (kKStep * 2) + ((c ^ (r & 7)) << 4);
}

template <int NB>
__global__ __launch_bounds__(kThreads) void lm_head_kernel(LmArgs a) {
  constexpr int RG = 32 * NB;                       // hidden rows per group
  constexpr int kStage = RG * kKStep * 2;           // LDS bytes per step
  constexpr int kRed = kWaves * RG * sizeof(State); // epilogue states
  constexpr int kLds = 2 * kStage > kRed ? 2 * kStage : kRed;
  __shared__ __attribute__((aligned(16))) char smem[kLds];

  // tiles in vocabulary-major order, row groups inner; workgroups of one
  // XCD (blockIdx % 8) take a contiguous range, so the row groups of a
  // vocabulary tile run on the same XCD and share its weights in L2
  const int n_tiles = a.n_vt * a.n_rg;
  const int per_xcd = (n_tiles + 7) / 8;
  const int tile = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (tile >= n_tiles) return;
  const int vt = tile / a.n_rg;
  const int rg = tile % a.n_rg;

  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int col = lane & 31;
  const int hf = lane >> 5;
  const int v_wave = vt * kVocabTile + wave * 32;   // first vocab row of wave
  const int row0 = rg * RG;                         // first hidden row

  // ---- weights: lane streams row v_wave + col, bytes 64*hf .. 64*hf+63 of
  // each 128-byte k step (rows past V re-read row V-1; masked later)
  const int vrow = min(v_wave + col, a.V - 1);
  const uint16_t* wp = a.w + static_cast<int64_t>(vrow) * a.Hd + hf * 32;
  const int nsteps = a.Hd / kKStep;
  u16x8_t wa[kPF][4];
  auto wload = [&](int s, u16x8_t (&r)[4]) {
    const uint16_t* p = wp + s * kKStep;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      r[j] = __builtin_nontemporal_load(
          reinterpret_cast<const u16x8_t*>(p + j * 8));
  };

  // ---- hidden rows: thread t moves 16-byte chunks t, t+512, ... of the
  // step's RG x 128 bytes (rows past R re-read row R-1; never written out)
  constexpr int kChunks = RG * 8;
  constexpr int kCPT = (kChunks + kThreads - 1) / kThreads;
  int h_src[kCPT], h_dst[kCPT];
  bool h_on[kCPT];
#pragma unroll
  for (int u = 0; u < kCPT; ++u) {
    const int g = threadIdx.x + u * kThreads;
    h_on[u] = g < kChunks;
    const int r = h_on[u] ? g / 8 : 0;
    const int c = g % 8;
    const int hr = min(row0 + r, a.R - 1);
    h_src[u] = hr * a.Hd + c * 8;        // element offset within step 0
    h_dst[u] = h_off(r, c);
  }
  u16x8_t hreg[kCPT];
  auto hload = [&](int s) {
#pragma unroll
    for (int u = 0; u < kCPT; ++u)
      if (h_on[u])
        hreg[u] = *reinterpret_cast<const u16x8_t*>(a.hidden + h_src[u] +
                                                    s * kKStep);
  };
  auto hstore = [&](char* sb) {
#pragma unroll
    for (int u = 0; u < kCPT; ++u)
      if (h_on[u]) *reinterpret_cast<u16x8_t*>(sb + h_dst[u]) = hreg[u];
  };

  floatx16_t acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[b][e] = 0.f;

  // prologue: weights of steps 0..PF-1 in flight, hidden step 0 in LDS,
  // hidden step 1 in registers
#pragma unroll
  for (int p = 0; p < kPF; ++p) wload(min(p, nsteps - 1), wa[p]);
  hload(0);
  hstore(smem);
  if (nsteps > 1) hload(1);
  __syncthreads();

  // step s: B fragments from LDS buffer s&1, A from register stage s%PF;
  // then the next hidden step goes to the other buffer and the stage is
  // refilled with step s+PF.  One barrier per step: the buffer written in
  // step s was last read in step s-1, before that step's barrier.
  auto step = [&](const int j, const int s) __attribute__((always_inline)) {
    const char* sb = smem + (j & 1) * kStage;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const bf16x8_t af = __builtin_bit_cast(bf16x8_t, wa[j % kPF][kk]);
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const bf16x8_t bfr = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const u16x8_t*>(
                          sb + h_off(b * 32 + col, hf * 4 + kk)));
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, bfr, acc[b], 0,
                                                         0, 0);
      }
    }
    wload(min(s + kPF, nsteps - 1), wa[j % kPF]);
    if (s + 1 < nsteps) {
      hstore(smem + ((j + 1) & 1) * kStage);
      if (s + 2 < nsteps) hload(s + 2);
    }
    __syncthreads();
  };
  constexpr int U = kPF % 2 == 0 ? kPF : 2 * kPF;
  const int nfull = nsteps / U * U;
  for (int s0 = 0; s0 < nfull; s0 += U) {
#pragma unroll
    for (int j = 0; j < U; ++j) step(j, s0 + j);
  }
#pragma unroll
  for (int j = 0; j < U - 1; ++j) {
    if (nfull + j >= nsteps) break;
    step(j, nfull + j);
  }

  // ---- epilogue: lane (col, hf) of row block b holds logits of hidden row
  // row0 + 32b + col at vocabulary rows v_wave + 8*(e/4) + 4*hf + e%4
  State* red = reinterpret_cast<State*>(smem);       // [kWaves][RG]
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    float x[16];
    int idx[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int v = v_wave + 8 * (e >> 2) + 4 * hf + (e & 3);
      idx[e] = v;
      x[e] = v < a.V ? acc[b][e] : kNegInf;
    }
    State st = empty_state();
    push_block(st, x, idx, a.c2);
    merge(st, shfl_xor_state(st, 32), a.c2);
    if (hf == 0) red[wave * RG + b * 32 + col] = st;
  }
  __syncthreads();
  if (threadIdx.x < RG) {
    const int r = threadIdx.x;
    State st = red[r];
    for (int w = 1; w < kWaves; ++w) merge(st, red[w * RG + r], a.c2);
    const int row = row0 + r;
    if (row < a.R) {
      if (a.n_vt == 1) finish(st, row, a.argmax, a.entropy, a.pmax);
      else a.ws[static_cast<int64_t>(row) * a.n_vt + vt] = st;
    }
  }
}

// Merge the vocabulary-tile states of each row, lanes over tiles.
__global__ __launch_bounds__(kWave) void lm_head_merge_kernel(LmArgs a) {
  const int row = blockIdx.x;
  State st = empty_state();
  const State* p = a.ws + static_cast<int64_t>(row) * a.n_vt;
  for (int t = lane_id(); t < a.n_vt; t += kWave) merge(st, p[t], a.c2);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1)
    merge(st, shfl_xor_state(st, off), a.c2);
  if (lane_id() == 0) finish(st, row, a.argmax, a.entropy, a.pmax);
}

// Rows per group: all R rows when R <= 128 (one pass over the weights),
// else groups of 128.
int blocks_per_wave(int R) {
  const int nb = (R + 31) / 32;
  return nb < 4 ? nb : 4;
}

bool lm_shape_ok(int R, int Hd, int V) {
  return R >= 1 && Hd >= kKStep && Hd % kKStep == 0 && V >= 1 &&
         static_cast<int64_t>(V) * Hd < (1ll << 40) &&
         static_cast<int64_t>(R) * Hd < (1ll << 31);
}

}  // namespace

extern "C" size_t wedlm_lm_head_score_workspace_size(int32_t R, int32_t Hd,
                                                     int32_t V) {
  if (!lm_shape_ok(R, Hd, V)) return 0;
  const int n_vt = (V + kVocabTile - 1) / kVocabTile;
  return n_vt > 1 ? static_cast<size_t>(R) * n_vt * sizeof(State) : 0;
}

extern "C" int wedlm_lm_head_score(const uint16_t* hidden,
                                   const uint16_t* w_vocab, int32_t R,
                                   int32_t Hd, int32_t V, double temperature,
                                   int32_t* argmax, float* entropy,
                                   float* pmax, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  if (!hidden || !w_vocab || !argmax || !entropy) return WEDLM_E_ARG;
  if (!(temperature > 0.0) || !(temperature < 1e30)) return WEDLM_E_ARG;
  if (!lm_shape_ok(R, Hd, V)) return WEDLM_E_SHAPE;
  const size_t need = wedlm_lm_head_score_workspace_size(R, Hd, V);
  if (workspace_bytes < need || (need && !workspace)) return WEDLM_E_WORKSPACE;
  LmArgs a{};
  a.hidden = hidden; a.w = w_vocab; a.R = R; a.Hd = Hd; a.V = V;
  a.n_vt = (V + kVocabTile - 1) / kVocabTile;
  const int nb = blocks_per_wave(R);
  a.n_rg = (R + 32 * nb - 1) / (32 * nb);
  a.c2 = 1.4426950408889634074 / temperature;
  a.argmax = argmax; a.entropy = entropy; a.pmax = pmax;
  a.ws = static_cast<State*>(workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t tiles = static_cast<int64_t>(a.n_vt) * a.n_rg;
  if (tiles > (1ll << 30)) return WEDLM_E_SHAPE;
  const unsigned grid = static_cast<unsigned>((tiles + 7) / 8 * 8);
  switch (nb) {
    case 1: hipLaunchKernelGGL(lm_head_kernel<1>, dim3(grid), dim3(kThreads), 0, st, a); break;
    case 2: hipLaunchKernelGGL(lm_head_kernel<2>, dim3(grid), dim3(kThreads), 0, st, a); break;
    case 3: hipLaunchKernelGGL(lm_head_kernel<3>, dim3(grid), dim3(kThreads), 0, st, a); break;
    default: hipLaunchKernelGGL(lm_head_kernel<4>, dim3(grid), dim3(kThreads), 0, st, a); break;
  }
  WEDLM_LAUNCH_CHECK();
  if (a.n_vt > 1) {
    hipLaunchKernelGGL(lm_head_merge_kernel, dim3(R), dim3(kWave), 0, st, a);
    WEDLM_LAUNCH_CHECK();
  }
  return WEDLM_OK;
}
