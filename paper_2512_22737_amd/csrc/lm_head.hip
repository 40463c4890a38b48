// LM head fused with the score of each row: logits = hidden . W_vocab^T on
// bf16 MFMA, reduced on the fly to the greedy token, entropy and top
// probability of softmax(logits / T) (Sec. 5.2; the Forward of Algorithm 1
// produces the logits the mask slots are scored on).  The fp32 logits are
// never written to memory.
//
// Up to 32 rows with Hd = 2048 or 4096 take lm_head_ks_kernel (the k split
// over the waves of a workgroup, described above it); every other shape the
// kernel below.
//
// Work decomposition (persistent, balanced):
//   grid      = n_rg row groups x n_slot slots, sized from the occupancy so
//               that every workgroup is resident at once
//   waves     = VW vocabulary waves x RW row waves (VW * RW = 8); vocabulary
//               wave v is stream j = slot*VW + v of its row group, which owns
//               the contiguous vocabulary range [j*V/S, (j+1)*V/S) (S = VW
//               n_slot streams), so ranges differ by at most one row; it
//               walks the range in blocks of 32*VB rows (VB = 1, or 2 for
//               the shapes with several row waves).  The RW row waves of a
//               stream take NB 32-row blocks of hidden rows each (a row
//               group is 32*NB*RW rows), read the same weights (fetched once
//               per CU, then from L1) and keep a running score state per row
//   MFMA      = v_mfma_f32_32x32x16_bf16 computing logits^T: A = 32 weight
//               rows x 16 k, B = 16 k x 32 hidden rows, both read from LDS;
//               a wave's step is VB x NB MFMAs per 16-wide k slice
//   k order   = the contraction runs over k in a permuted order that is the
//               same for A and B: in each 64-wide k step, lane half hf of
//               MFMA j takes k = 32*hf + 8*j .. +8, i.e. 16-byte chunk
//               4*hf + j of a 128-byte LDS row, for both operands.
// Memory path: the weights are the HBM stream (V * Hd * 2 bytes per row
//   group).  A stream's 32*VB rows of a k step (4 KB per 32 rows) are
//   loaded coalesced, eight full 128-byte rows per wave instruction, split
//   over its row waves, PF steps ahead across block boundaries, and go
//   through a double-buffered LDS tile of the stream (a pattern with one
//   row per lane touches 32 lines per instruction and streams about 25%
//   slower).  The hidden rows of a step go through LDS the same way
//   (groups beyond 384 rows load both straight into LDS instead:
//   lm_head_dma_kernel).  All LDS rows are XOR-swizzled 16-byte chunks;
//   one barrier per step orders every buffer.
//   Slots are placed so that the row groups of one slot share an XCD (and
//   the weights they stream in its L2).
// Epilogue: after each block a lane holds 16 logits of one hidden row per
//   row block; they enter the wave's running state (score_state.h), merged
//   across the two lane halves; at the end the eight waves merge in LDS and
//   the slots in a merge kernel over a workspace of per-slot states.
// Roofline: 2 * R * Hd * V flops against V * Hd * 2 weight bytes per row
//   group; R rows in one group give an intensity of R flop/byte.
#include <algorithm>

#include "common.h"
#include "score_state.h"

using namespace wedlm;

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * kWave;
constexpr int kKStep = 64;                // k per pipeline step
constexpr int kPF = 4;                    // weight steps in flight per wave

struct LmArgs {
  const uint16_t* hidden;   // [R, Hd]
  const uint16_t* w;        // [V, Hd]
  int R, Hd, V;
  int n_rg, n_slot;         // row groups, slots (per row group)
  int nblk;                 // 32-row vocabulary blocks per stream
  double c2;                // log2(e) / T
  int32_t* argmax;
  float* entropy;
  float* pmax;
  State* ws;                // [R, n_slot] (n_slot > 1)
};

// LDS row of one k step: 64 bf16 = eight 16-byte chunks; chunk c of row r
// sits in slot c ^ (r & 7), so the 8 lanes of one ds_read_b128 pass (8 rows,
// same chunk) hit 8 different slots.
__device__ __forceinline__ int h_off(int r, int c) {
  return r * (kKStep * 2) + ((c ^ (r & 7)) << 4);
}

// NB 32-row blocks of hidden rows per wave, RW row waves, VB 32-row
// vocabulary blocks per wave and step, HPF register stages of hidden rows
// (a divisor of kPF); NT: weight loads carry the
// non-temporal hint (one row group: nothing else reads the lines; with
// several, the groups share them through L2 and the hint costs 5%)
template <int NB, int RW, int HPF, bool NT, int VB = 1>
__global__ __launch_bounds__(kThreads) void lm_head_kernel(LmArgs a) {
  constexpr int VW = kWaves / RW;                   // vocabulary waves
  constexpr int RB = 32 * NB;                       // hidden rows per wave
  constexpr int RG = RB * RW;                       // hidden rows per group
  constexpr int BR = 32 * VB;                       // vocabulary rows per block
  constexpr int NJ = 4 * VB / RW;                   // weight loads per wave
  static_assert(kWaves % RW == 0 && (4 * VB) % RW == 0 && kPF % HPF == 0,
                "wave and stage split");
  constexpr int kStage = RG * kKStep * 2;           // hidden LDS per step
  constexpr int kWTile = BR * kKStep * 2;           // weight LDS per step
  constexpr int kWBase = 2 * kStage;                // weight tiles after
  constexpr int kRed = kWaves * RB * sizeof(State); // epilogue states
  constexpr int kMain = kWBase + VW * 2 * kWTile;
  constexpr int kLds = kMain > kRed ? kMain : kRed;
  __shared__ __attribute__((aligned(16))) char smem[kLds];

  const int xcd = blockIdx.x % 8;
  const int local = blockIdx.x / 8;
  const int rg = local % a.n_rg;
  const int slot = (local / a.n_rg) * 8 + xcd;
  if (slot >= a.n_slot) return;

  const int wave = threadIdx.x / kWave;
  const int vw = wave % VW;
  const int rw = wave / VW;
  const int lane = lane_id();
  const int col = lane & 31;
  const int hf = lane >> 5;
  const int row0 = rg * RG;                         // first hidden row
  const int64_t S = static_cast<int64_t>(a.n_slot) * VW;
  const int64_t j = static_cast<int64_t>(slot) * VW + vw;
  const int v_lo = static_cast<int>(j * a.V / S);
  const int v_hi = static_cast<int>((j + 1) * a.V / S);
  const int nsteps = a.Hd / kKStep;                 // a multiple of kPF
  const int nblk = a.nblk;
  const int total = nblk * nsteps;

  // ---- weights: the stream's BR rows x 128 bytes of a k step are 4*VB
  // 1 KB loads (8 rows each, lane l: row l/8 + 8j, chunk l%8); row wave rw
  // issues loads j = rw, rw+RW, ...  Every load is issued (no branch in the
  // step, so the compiler's waits stay partial): a row past the stream's
  // range re-reads its last row and its logits are masked; steps past the
  // end re-read the last.
  const int v_last = max(v_hi - 1, 0);
  const int w_row = lane >> 3, w_chunk = lane & 7;
  char* const wtile = smem + kWBase + vw * 2 * kWTile;   // [2][BR x 128 B]
  u16x8_t wa[kPF][NJ];
  auto wload = [&](int q, u16x8_t (&r)[NJ]) {
    q = min(q, total - 1);
    const int bi = q / nsteps;
    const int s = q - bi * nsteps;
#pragma unroll
    for (int i = 0; i < NJ; ++i) {
      const int rr = w_row + 8 * (rw + i * RW);
      const int v = min(v_lo + BR * bi + rr, v_last);
      const u16x8_t* p = reinterpret_cast<const u16x8_t*>(
          a.w + static_cast<int64_t>(v) * a.Hd + s * kKStep + w_chunk * 8);
      if constexpr (NT)
        r[i] = __builtin_nontemporal_load(p);
      else
        r[i] = *p;
    }
  };
  auto wstore = [&](char* wb, const u16x8_t (&r)[NJ]) {
#pragma unroll
    for (int i = 0; i < NJ; ++i)
      *reinterpret_cast<u16x8_t*>(wb + h_off(w_row + 8 * (rw + i * RW),
                                             w_chunk)) = r[i];
  };

  // ---- hidden rows: thread t moves 16-byte chunks t, t+512, ... of the
  // step's RG x 128 bytes, modulo RG*8 (when RG*8 < 512 two threads write the
  // same chunk with the same bytes); rows past R re-read row R-1 and are
  // never written out
  constexpr int kChunks = RG * 8;
  constexpr int kCPT = (kChunks + kThreads - 1) / kThreads;
  int h_src[kCPT], h_dst[kCPT];
#pragma unroll
  for (int u = 0; u < kCPT; ++u) {
    const int g = (threadIdx.x + u * kThreads) % kChunks;
    const int r = g / 8;
    const int c = g % 8;
    const int hr = min(row0 + r, a.R - 1);
    h_src[u] = hr * a.Hd + c * 8;        // element offset within step 0
    h_dst[u] = h_off(r, c);
  }
  // a ring of HPF register stages: step s's rows live in stage s % HPF,
  // loaded HPF steps before they go to LDS (L2 latency hidden)
  u16x8_t hreg[HPF][kCPT];
  auto hload = [&](int s, u16x8_t (&r)[kCPT]) {
#pragma unroll
    for (int u = 0; u < kCPT; ++u)
      r[u] = *reinterpret_cast<const u16x8_t*>(a.hidden + h_src[u] +
                                               s * kKStep);
  };
  auto hstore = [&](char* sb, const u16x8_t (&r)[kCPT]) {
#pragma unroll
    for (int u = 0; u < kCPT; ++u)
      *reinterpret_cast<u16x8_t*>(sb + h_dst[u]) = r[u];
  };
  auto hstep = [&](int s) { return ((s % nsteps) + nsteps) % nsteps; };

  floatx16_t acc[VB][NB];
  auto zero_acc = [&]() {
#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[vb][b][e] = 0.f;
  };
  zero_acc();
  State st[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) st[b] = empty_state();
  const ExpScale sc = exp_scale(a.c2);

  // prologue: step 0's hidden rows and weights into LDS, then the loads of
  // the PF steps before step 0 issued as those steps would (weights of step
  // p+1 into stage (p+1) % PF, then hidden step p - PF + 1 + HPF into its
  // stage; steps before 0 wrap and are never used), so the loop head sees
  // the same loads in flight from both of its predecessors and the
  // compiler's waits stay partial
  hload(0, hreg[0]);
  wload(0, wa[0]);
  hstore(smem, hreg[0]);
  wstore(wtile, wa[0]);
#pragma unroll
  for (int p = 0; p < kPF; ++p) {
    wload(p + 1, wa[(p + 1) % kPF]);
    const int hs = p - kPF + 1 + HPF;
    hload(hstep(hs), hreg[((hs % HPF) + HPF) % HPF]);
  }
  __syncthreads();

  // step q = bi*nsteps + s (u = s % kPF, static): A and B fragments from
  // the LDS buffers s&1 (nsteps is even); then step s+1's weights (register
  // stage (u+1) % PF) and hidden rows (stage (u+1) % HPF) go to the other
  // buffers and those stages are refilled with steps q+1+PF and s+1+HPF
  // (unconditionally: past the last step these are re-reads nobody uses).
  // One barrier per step: a buffer written in step q was last read in step
  // q-1, before its barrier, and is read in step q+1, after this one.
  auto step = [&](const int u, const int q, const int s)
      __attribute__((always_inline)) {
    const char* sb = smem + (u & 1) * kStage;
    const char* wb = wtile + (u & 1) * kWTile;
    // fragments of all four k slices read up front (one slice at a time
    // with two vocabulary blocks per wave, for registers)
    constexpr int KF = VB == 1 ? 4 : 1;
#pragma unroll
    for (int k0 = 0; k0 < 4; k0 += KF) {
      bf16x8_t afr[KF][VB];
#pragma unroll
      for (int kk = 0; kk < KF; ++kk)
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
          afr[kk][vb] = __builtin_bit_cast(
              bf16x8_t, *reinterpret_cast<const u16x8_t*>(
                            wb + h_off(vb * 32 + col, hf * 4 + k0 + kk)));
      bf16x8_t bfr[KF][NB];
#pragma unroll
      for (int kk = 0; kk < KF; ++kk)
#pragma unroll
        for (int b = 0; b < NB; ++b)
          bfr[kk][b] = __builtin_bit_cast(
              bf16x8_t,
              *reinterpret_cast<const u16x8_t*>(
                  sb + h_off(rw * RB + b * 32 + col, hf * 4 + k0 + kk)));
#pragma unroll
      for (int kk = 0; kk < KF; ++kk) {
#pragma unroll
        for (int vb = 0; vb < VB; ++vb)
#pragma unroll
          for (int b = 0; b < NB; ++b)
            acc[vb][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                afr[kk][vb], bfr[kk][b], acc[vb][b], 0, 0, 0);
      }
    }
    wstore(wtile + ((u + 1) & 1) * kWTile, wa[(u + 1) % kPF]);
    wload(q + 1 + kPF, wa[(u + 1) % kPF]);
    hstore(smem + ((u + 1) & 1) * kStage, hreg[(u + 1) % HPF]);
    hload(hstep(s + 1 + HPF), hreg[(u + 1) % HPF]);
    __syncthreads();
  };

  for (int bi = 0; bi < nblk; ++bi) {
    for (int s0 = 0; s0 < nsteps; s0 += kPF) {
#pragma unroll
      for (int u = 0; u < kPF; ++u)
        step(u, bi * nsteps + s0 + u, s0 + u);
    }
    // block done: lane (col, hf) of row block b holds logits of hidden row
    // row0 + RB*rw + 32b + col at vocabulary rows
    // v0 + 32*vb + 8*(e/4) + 4*hf + e%4
    const int v0 = v_lo + BR * bi;
#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        float x[16];
        int idx[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int v = v0 + 32 * vb + 8 * (e >> 2) + 4 * hf + (e & 3);
          idx[e] = v;
          x[e] = v < v_hi ? acc[vb][b][e] : kNegInf;
        }
        push_block(st[b], x, idx, sc);
      }
    zero_acc();
  }

  // ---- the waves' states: both lane halves, then the VW vocabulary waves
  // of each row wave in LDS
  State* red = reinterpret_cast<State*>(smem);       // [kWaves][RB]
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    merge(st[b], shfl_xor_state(st[b], 32), a.c2);
    if (hf == 0) red[wave * RB + b * 32 + col] = st[b];
  }
  __syncthreads();
  if (threadIdx.x < RG) {
    const int r = threadIdx.x;
    const int r_w = r / RB, r_l = r % RB;            // row wave, its row
    State m = red[(r_w * VW) * RB + r_l];
    for (int v = 1; v < VW; ++v) merge(m, red[(r_w * VW + v) * RB + r_l], a.c2);
    const int row = row0 + r;
    if (row < a.R) {
      if (a.n_slot == 1) finish(m, row, a.argmax, a.entropy, a.pmax);
      else a.ws[static_cast<int64_t>(row) * a.n_slot + slot] = m;
    }
  }
}

// Large row groups: the same decomposition, but a step's hidden rows and
// weights go from memory straight into one of two LDS stages with
// LDS-destination buffer loads (lane l of a 1 KB load lands at LDS row l/8,
// slot l%8, so it fetches the chunk (l%8) ^ (l/8) that the XOR swizzle puts
// there).  With no register staging a wave can hold 64 vocabulary x 128
// hidden rows of accumulators (NB 4, RW 4, VB 2: a 512-row group, one pass
// over the weights, 0.75 KB of LDS reads per MFMA).  The loads of step q+1
// are issued before step q computes and waited for before the barrier that
// ends it.  Weights are read through a buffer resource over the stream's
// own rows, hidden rows through one over the group's rows (reads past them
// return zero; rows past the range are clamped to its last one and their
// logits masked), so every offset is that of a few megabytes.
template <int NB, int RW, int VB, bool NT>
__global__ __launch_bounds__(kThreads) void lm_head_dma_kernel(LmArgs a) {
  constexpr int VW = kWaves / RW;
  constexpr int RB = 32 * NB;
  constexpr int RG = RB * RW;
  constexpr int BR = 32 * VB;
  constexpr int kHStage = RG * kKStep * 2;
  constexpr int kWTileB = BR * kKStep * 2;
  constexpr int kStageB = kHStage + VW * kWTileB;
  constexpr int kHLoads = RG / 8 / kWaves;
  constexpr int kWLoads = BR / 8 / RW;
  static_assert(RG % (8 * kWaves) == 0 && BR % (8 * RW) == 0, "load split");
  constexpr int kRed = kWaves * RB * sizeof(State);
  constexpr int kLds = 2 * kStageB > kRed ? 2 * kStageB : kRed;
  __shared__ __attribute__((aligned(1024))) char smem[kLds];

  const int xcd = blockIdx.x % 8;
  const int local = blockIdx.x / 8;
  const int rg = local % a.n_rg;
  const int slot = (local / a.n_rg) * 8 + xcd;
  if (slot >= a.n_slot) return;

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int vw = wave % VW;
  const int rw = wave / VW;
  const int lane = lane_id();
  const int col = lane & 31;
  const int hf = lane >> 5;
  const int row0 = rg * RG;
  const int64_t S = static_cast<int64_t>(a.n_slot) * VW;
  const int64_t j = static_cast<int64_t>(slot) * VW + vw;
  const int v_lo = static_cast<int>(j * a.V / S);
  const int v_hi = static_cast<int>((j + 1) * a.V / S);
  const int nsteps = a.Hd / kKStep;
  const int nblk = a.nblk;
  const int total = nblk * nsteps;

  const int lr = lane >> 3;
  const int lc = (lane & 7) ^ lr;
  const int w_rows = max(v_hi - v_lo, 1);
  const i32x4_t wrs = buffer_rsrc(a.w + static_cast<int64_t>(v_lo) * a.Hd,
                                  (v_hi - v_lo) * a.Hd * 2);
  const int h_rows = min(a.R - row0, RG);
  const i32x4_t hrs = buffer_rsrc(a.hidden + static_cast<int64_t>(row0) * a.Hd,
                                  h_rows * a.Hd * 2);
  const uint32_t lds0 =
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_t*)smem));
  auto issue = [&](int q, int stage) {
    q = min(q, total - 1);
    const int bi = q / nsteps;
    const int s = q - bi * nsteps;
#pragma unroll
    for (int i = 0; i < kHLoads; ++i) {
      const int blk = wave + kWaves * i;
      const int r = min(8 * blk + lr, h_rows - 1);
      load_to_lds16<false>(hrs, r * a.Hd * 2 + s * 128 + lc * 16,
                           __builtin_amdgcn_readfirstlane(
                               lds0 + stage * kStageB + blk * 1024));
    }
#pragma unroll
    for (int i = 0; i < kWLoads; ++i) {
      const int blk = rw + RW * i;
      const int rr = min(BR * bi + 8 * blk + lr, w_rows - 1);
      load_to_lds16<NT>(wrs, rr * a.Hd * 2 + s * 128 + lc * 16,
                        __builtin_amdgcn_readfirstlane(
                            lds0 + stage * kStageB + kHStage + vw * kWTileB +
                            blk * 1024));
    }
  };

  floatx16_t acc[VB][NB];
  auto zero_acc = [&]() {
#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[vb][b][e] = 0.f;
  };
  zero_acc();
  State st[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) st[b] = empty_state();
  const ExpScale sc = exp_scale(a.c2);

  auto compute = [&](int buf) __attribute__((always_inline)) {
    const char* sb = smem + buf * kStageB;
    const char* wb = sb + kHStage + vw * kWTileB;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      bf16x8_t afr[VB], bfr[NB];
#pragma unroll
      for (int vb = 0; vb < VB; ++vb)
        afr[vb] = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const u16x8_t*>(
                          wb + h_off(vb * 32 + col, hf * 4 + kk)));
#pragma unroll
      for (int b = 0; b < NB; ++b)
        bfr[b] = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const u16x8_t*>(
                          sb + h_off(rw * RB + b * 32 + col, hf * 4 + kk)));
#pragma unroll
      for (int vb = 0; vb < VB; ++vb)
#pragma unroll
        for (int b = 0; b < NB; ++b)
          acc[vb][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              afr[vb], bfr[b], acc[vb][b], 0, 0, 0);
    }
  };

  issue(0, 0);
  wait_vmcnt<0>();
  __syncthreads();
  for (int bi = 0; bi < nblk; ++bi) {
    for (int s = 0; s < nsteps; ++s) {
      const int q = bi * nsteps + s;
      issue(q + 1, (q + 1) & 1);
      compute(q & 1);
      wait_vmcnt<0>();
      __syncthreads();
    }
    const int v0 = v_lo + BR * bi;
#pragma unroll
    for (int vb = 0; vb < VB; ++vb)
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        float x[16];
        int idx[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int v = v0 + 32 * vb + 8 * (e >> 2) + 4 * hf + (e & 3);
          idx[e] = v;
          x[e] = v < v_hi ? acc[vb][b][e] : kNegInf;
        }
        push_block(st[b], x, idx, sc);
      }
    zero_acc();
  }

  State* red = reinterpret_cast<State*>(smem);
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    merge(st[b], shfl_xor_state(st[b], 32), a.c2);
    if (hf == 0) red[wave * RB + b * 32 + col] = st[b];
  }
  __syncthreads();
  if (threadIdx.x < RG) {
    const int r = threadIdx.x;
    const int r_w = r / RB, r_l = r % RB;
    State m = red[(r_w * VW) * RB + r_l];
    for (int v = 1; v < VW; ++v) merge(m, red[(r_w * VW + v) * RB + r_l], a.c2);
    const int row = row0 + r;
    if (row < a.R) {
      if (a.n_slot == 1) finish(m, row, a.argmax, a.entropy, a.pmax);
      else a.ws[static_cast<int64_t>(row) * a.n_slot + slot] = m;
    }
  }
}

// Few rows (R <= 32): the k split over the waves.  A workgroup of NWV
// waves owns a contiguous run of 32-row vocabulary blocks (the runs of the
// grid differ by at most one block); wave w owns the k steps w, w + NWV,
// w + 2 NWV, ... of every block, so at any time the workgroup reads NWV
// neighbouring 128-byte pieces of each of the block's 32 rows.  The wave's
// hidden-row fragments of its k steps stay in registers for the whole run
// (SPW steps x 4 MFMAs); its weight rows go through a private
// double-buffered 4 KB LDS tile per k step (loaded coalesced, eight full
// 128-byte rows per instruction, PF steps ahead across block boundaries),
// so the loop needs no barrier.  After each block the NWV partial 32 x 32
// logit tiles are summed through LDS in wave order (one barrier; two
// buffers alternate between blocks) and wave w scores 16 / NWV of the 16
// vocabulary rows each lane holds.
// Measured at Hd 4096, V 151936 (R = 16 and 32): 207 us, 6.0 TB/s, where
// the vocabulary split over 2048 wave streams (74 rows each) took 236-245
// us; with four waves and a contiguous k range per wave (each reading 2 KB
// apart in every row) the k split took 285 us, and more vocabulary streams
// made the other kernel slower, not faster: the number of scattered
// streams in flight, not padding, set its rate.
constexpr int kKsWaves = 8;
constexpr int kKsPF = 4;   // register stages of weight steps in flight

template <int SPW, int PF>
__global__ __launch_bounds__(kKsWaves * kWave) void lm_head_ks_kernel(LmArgs a) {
  constexpr int NWV = kKsWaves;
  constexpr int EPW = 16 / NWV;                            // entries per wave
  static_assert(SPW % PF == 0 && (SPW & 1) == 0, "stages line up with blocks");
  static_assert(EPW == 2 || EPW == 4, "waves");
  constexpr int kWTile = 32 * kKStep * 2;                  // 4 KB
  constexpr int kRedBuf = NWV * 16 * kWave * 4;
  __shared__ __attribute__((aligned(16))) char smem[NWV * 2 * kWTile + 2 * kRedBuf];
  const int wave = threadIdx.x / kWave;
  const int lane = lane_id();
  const int col = lane & 31;
  const int hf = lane >> 5;
  const int g = blockIdx.x;
  const int nba = (a.V + 31) / 32;
  const int bb0 = static_cast<int>(static_cast<int64_t>(g) * nba / a.n_slot);
  const int bb1 = static_cast<int>(static_cast<int64_t>(g + 1) * nba / a.n_slot);
  const int nblk = bb1 - bb0;
  const int total = nblk * SPW;

  // hidden-row fragments of this wave's k steps (rows past R re-read R-1)
  const uint16_t* hrow =
      a.hidden + static_cast<int64_t>(min(col, a.R - 1)) * a.Hd + hf * 32;
  bf16x8_t bfr[SPW][4];
#pragma unroll
  for (int s = 0; s < SPW; ++s)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      bfr[s][j] = __builtin_bit_cast(
          bf16x8_t, *reinterpret_cast<const u16x8_t*>(
                        hrow + (s * NWV + wave) * kKStep + j * 8));

  // weights: 32 rows x 128 bytes of a k step as four 1 KB loads (lane l:
  // row l/8 + 8i, chunk l%8); rows past V re-read row V-1 (masked later),
  // steps past the run re-read its last step
  const int w_row = lane >> 3, w_chunk = lane & 7;
  char* const wtile = smem + wave * 2 * kWTile;
  auto wload = [&](int q, u16x8_t (&r)[4]) {
    q = min(q, total - 1);
    const int bi = q / SPW;
    const int s = q - bi * SPW;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = min((bb0 + bi) * 32 + w_row + 8 * i, a.V - 1);
      r[i] = __builtin_nontemporal_load(reinterpret_cast<const u16x8_t*>(
          a.w + static_cast<int64_t>(v) * a.Hd + (s * NWV + wave) * kKStep +
          w_chunk * 8));
    }
  };
  auto wstore = [&](char* wb, const u16x8_t (&r)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<u16x8_t*>(wb + h_off(w_row + 8 * i, w_chunk)) = r[i];
  };

  floatx16_t acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.f;
  State st = empty_state();
  const ExpScale sc = exp_scale(a.c2);
  float* const red = reinterpret_cast<float*>(smem + NWV * 2 * kWTile);

  u16x8_t wa[PF][4];
  if (nblk > 0) {
    wload(0, wa[0]);
    wstore(wtile, wa[0]);
#pragma unroll
    for (int p = 0; p < PF; ++p) wload(p + 1, wa[(p + 1) % PF]);
  }
  for (int bi = 0; bi < nblk; ++bi) {
#pragma unroll
    for (int s = 0; s < SPW; ++s) {
      const int q = bi * SPW + s;
      const int u = s % PF;                                // = q % PF
      const char* wb = wtile + (s & 1) * kWTile;           // SPW is even
      bf16x8_t afr[4];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        afr[kk] = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const u16x8_t*>(wb + h_off(col, hf * 4 + kk)));
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(afr[kk], bfr[s][kk], acc,
                                                       0, 0, 0);
      wstore(wtile + ((s + 1) & 1) * kWTile, wa[(u + 1) % PF]);
      wload(q + 1 + PF, wa[(u + 1) % PF]);
    }
    // partial tiles -> LDS [buffer][wave][e/4][lane] (16 bytes per entry)
    float* rb = red + (bi & 1) * (kRedBuf / 4);
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4) {
      const floatx4_t v = {acc[4 * e4], acc[4 * e4 + 1], acc[4 * e4 + 2],
                           acc[4 * e4 + 3]};
      *reinterpret_cast<floatx4_t*>(rb + ((wave * 4 + e4) * kWave + lane) * 4) = v;
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.f;
    __syncthreads();
    // wave w: entries e = EPW*w .. EPW*w + EPW-1, summed over the waves in
    // order; entry e of lane (col, hf) is vocabulary row 8(e/4) + 4hf + e%4
    const int e0 = wave * EPW;
    float sum[EPW];
#pragma unroll
    for (int t = 0; t < EPW; ++t) sum[t] = 0.f;
#pragma unroll
    for (int w2 = 0; w2 < NWV; ++w2) {
      const float* src = rb + ((w2 * 4 + e0 / 4) * kWave + lane) * 4 + e0 % 4;
#pragma unroll
      for (int t = 0; t < EPW; ++t) sum[t] += src[t];
    }
    const int v0 = (bb0 + bi) * 32 + 8 * (e0 / 4) + 4 * hf + e0 % 4;
    float x[EPW];
    int idx[EPW];
#pragma unroll
    for (int t = 0; t < EPW; ++t) {
      idx[t] = v0 + t;
      x[t] = v0 + t < a.V ? sum[t] : kNegInf;
    }
    push_block(st, x, idx, sc);
  }

  // merge: the two lane halves, then the waves (LDS, after a barrier)
  merge(st, shfl_xor_state(st, 32), a.c2);
  __syncthreads();
  State* sred = reinterpret_cast<State*>(red);            // [wave][32]
  if (hf == 0) sred[wave * 32 + col] = st;
  __syncthreads();
  if (threadIdx.x < 32 && threadIdx.x < a.R) {
    const int r = threadIdx.x;
    State m = sred[r];
    for (int w2 = 1; w2 < NWV; ++w2) merge(m, sred[w2 * 32 + r], a.c2);
    if (a.n_slot == 1) finish(m, r, a.argmax, a.entropy, a.pmax);
    else a.ws[static_cast<int64_t>(r) * a.n_slot + g] = m;
  }
}

// Merge the slot states of each row, lanes over slots.
__global__ __launch_bounds__(kWave) void lm_head_merge_kernel(LmArgs a) {
  const int row = blockIdx.x;
  State st = empty_state();
  const State* p = a.ws + static_cast<int64_t>(row) * a.n_slot;
  for (int t = lane_id(); t < a.n_slot; t += kWave) merge(st, p[t], a.c2);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1)
    merge(st, shfl_xor_state(st, off), a.c2);
  if (lane_id() == 0) finish(st, row, a.argmax, a.entropy, a.pmax);
}

// Row groups: up to 96 rows, one row wave with 1..3 blocks (a 256 x R
// tile); 97..128 rows, two row waves of 2 blocks; 129..256 rows, four row
// waves of 2 blocks; 257..384 rows, four row waves of 3 blocks; beyond,
// groups of 512 rows in four row waves of 4 blocks (lm_head_dma_kernel).
// The multi-wave shapes give each wave two 32-row vocabulary blocks, so a
// 64-row vocabulary tile feeds every hidden-row fragment twice: the loop
// is bound by LDS reads, and this takes them from 1.25 KB per MFMA (one
// vocabulary block, four row blocks) to 1.0 (2 x 2), 0.83 (2 x 3) and
// 0.75 (2 x 4).  Measured against one vocabulary block per wave: 9% faster
// at 128 rows, 6% at 256, 17% at 384 (one group of 384 rows against two of
// 192).  The 512-row groups need the register-free staging of the DMA
// kernel (128 accumulator registers) and against 256-row groups measured
// 14% faster at 448 and 512 rows, 39% at 768 and 12% at 1024; at 384 rows
// the DMA kernel with 3 blocks ties the register-staged one.
struct Shape {
  int nb, rw;
  int vb = 1;             // 32-row vocabulary blocks per wave and step
  bool dma = false;       // lm_head_dma_kernel
};

Shape group_shape(int R) {
  if (R <= 96) return {(R + 31) / 32, 1};
  if (R <= 128) return {2, 2, 2};
  if (R <= 256) return {2, 4, 2};
  if (R <= 384) return {3, 4, 2};
  return {4, 4, 2, true};
}

// Hd a multiple of 4 k steps: the weight stages then line up with the steps
// of every block.
bool lm_shape_ok(int R, int Hd, int V) {
  return R >= 1 && Hd >= kKStep * kPF && Hd % (kKStep * kPF) == 0 && V >= 1 &&
         static_cast<int64_t>(V) * Hd < (1ll << 40) &&
         static_cast<int64_t>(R) * Hd < (1ll << 31);
}

template <int NB, int RW, int HPF, int VB = 1>
int resident_per_cu() {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &n,
          reinterpret_cast<const void*>(lm_head_kernel<NB, RW, HPF, true, VB>),
          kThreads, 0) != hipSuccess || n < 1)
    n = 1;
  return n;
}

// the kernel of each group shape; occupancy index 0..5
constexpr int kShapes = 7;
int shape_index(Shape s) {
  if (s.dma) return 6;
  if (s.vb == 1) return s.nb - 1;
  return s.rw == 2 ? 3 : s.nb == 2 ? 4 : 5;
}

// Slots per row group: every workgroup resident at once (CUs x occupancy),
// no more streams than 32-row blocks.  Cached per device.
struct LmPlan {
  Shape sh;
  int n_rg, n_slot, nblk;
  int ks_spw;   // > 0: the k-split kernel with this many k steps per wave
};

// The k-split kernel takes R <= 32 rows and Hd = 2048 or 4096 (k steps per
// wave a compile-time count).
int ks_steps_per_wave(int R, int Hd) {
  if (R > 32 || Hd % (kKStep * kKsWaves) != 0) return 0;
  const int spw = Hd / kKStep / kKsWaves;
  return spw == 4 || spw == 8 ? spw : 0;
}

template <int SPW>
int ks_resident_per_cu() {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &n, reinterpret_cast<const void*>(lm_head_ks_kernel<SPW, kKsPF>),
          kKsWaves * kWave, 0) != hipSuccess || n < 1)
    n = 1;
  return n;
}

template <int NB, int RW, int VB>
int dma_resident_per_cu() {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &n, reinterpret_cast<const void*>(lm_head_dma_kernel<NB, RW, VB, true>),
          kThreads, 0) != hipSuccess || n < 1)
    n = 1;
  return n;
}
template <int NB, int RW, int VB>
void launch_dma(bool nt, int64_t grid, hipStream_t st, const LmArgs& a) {
  if (nt)
    hipLaunchKernelGGL((lm_head_dma_kernel<NB, RW, VB, true>), dim3(grid),
                       dim3(kThreads), 0, st, a);
  else
    hipLaunchKernelGGL((lm_head_dma_kernel<NB, RW, VB, false>), dim3(grid),
                       dim3(kThreads), 0, st, a);
}

bool lm_plan(int R, int Hd, int V, LmPlan* p) {
  if (!lm_shape_ok(R, Hd, V)) return false;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return false;
  static int cus[64], occ[64][kShapes], occ_ks[64][2];
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount,
                              dev) != hipSuccess || n < 1)
      return false;
    occ[dev][0] = resident_per_cu<1, 1, kPF>();
    occ[dev][1] = resident_per_cu<2, 1, kPF>();
    occ[dev][2] = resident_per_cu<3, 1, 2>();
    occ[dev][3] = resident_per_cu<2, 2, 2, 2>();
    occ[dev][4] = resident_per_cu<2, 4, 2, 2>();
    occ[dev][5] = resident_per_cu<3, 4, 1, 2>();
    occ[dev][6] = dma_resident_per_cu<4, 4, 2>();
    occ_ks[dev][0] = ks_resident_per_cu<4>();
    occ_ks[dev][1] = ks_resident_per_cu<8>();
    cus[dev] = n;
  }
  p->ks_spw = ks_steps_per_wave(R, Hd);
  if (p->ks_spw > 0) {
    const int oi = p->ks_spw == 4 ? 0 : 1;
    const int nba = (V + 31) / 32;
    p->sh = Shape{1, 1};
    p->n_rg = 1;
    p->n_slot = std::min(cus[dev] * occ_ks[dev][oi], nba);
    p->nblk = 0;
    return true;
  }
  auto slots = [&](Shape sh) {
    p->sh = sh;
    const int rg = 32 * sh.nb * sh.rw;
    const int vw = kWaves / sh.rw;
    const int br = 32 * sh.vb;
    p->n_rg = (R + rg - 1) / rg;
    int n_slot = cus[dev] * occ[dev][shape_index(sh)] / p->n_rg;
    const int by_blocks = (V + br * vw - 1) / (br * vw);
    if (n_slot > by_blocks) n_slot = by_blocks;
    if (n_slot < 1) n_slot = 1;
    p->n_slot = n_slot;
    const int64_t S = static_cast<int64_t>(n_slot) * vw;
    const int64_t per = (V + S - 1) / S;             // rows of the longest
    p->nblk = static_cast<int>((per + br - 1) / br);
    return per;
  };
  const Shape sh = group_shape(R);
  const int64_t per = slots(sh);
  // the DMA kernel's buffer resources hold 32-bit byte counts: a stream's
  // weight rows and a group's hidden rows must stay under 2 GiB
  if (sh.dma && (per * Hd * 2 >= (1ll << 31) ||
                 static_cast<int64_t>(32 * sh.nb * sh.rw) * Hd * 2 >= (1ll << 31)))
    slots(Shape{2, 4, 2});
  return true;
}

// groups of fewer than 128 rows only occur with R < 128: one group
// only the 256-row shape ever serves several row groups (nt false)
template <int NB, int RW, int HPF, int VB = 1>
void launch(bool nt, int64_t grid, hipStream_t st, const LmArgs& a) {
  if constexpr (32 * NB * RW != 256) {
    hipLaunchKernelGGL((lm_head_kernel<NB, RW, HPF, true, VB>), dim3(grid),
                       dim3(kThreads), 0, st, a);
  } else {
    if (nt)
      hipLaunchKernelGGL((lm_head_kernel<NB, RW, HPF, true, VB>), dim3(grid),
                         dim3(kThreads), 0, st, a);
    else
      hipLaunchKernelGGL((lm_head_kernel<NB, RW, HPF, false, VB>), dim3(grid),
                         dim3(kThreads), 0, st, a);
  }
}

}  // namespace

extern "C" size_t wedlm_lm_head_score_workspace_size(int32_t R, int32_t Hd,
                                                     int32_t V) {
  LmPlan p;
  if (!lm_plan(R, Hd, V, &p)) return 0;
  return p.n_slot > 1 ? static_cast<size_t>(R) * p.n_slot * sizeof(State) : 0;
}

extern "C" int wedlm_lm_head_score(const uint16_t* hidden,
                                   const uint16_t* w_vocab, int32_t R,
                                   int32_t Hd, int32_t V, double temperature,
                                   int32_t* argmax, float* entropy,
                                   float* pmax, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  if (!hidden || !w_vocab || !argmax || !entropy) return WEDLM_E_ARG;
  if (!(temperature > 0.0) || !(temperature < 1e30)) return WEDLM_E_ARG;
  LmPlan p;
  if (!lm_shape_ok(R, Hd, V)) return WEDLM_E_SHAPE;
  if (!lm_plan(R, Hd, V, &p)) return WEDLM_E_DEVICE;
  const size_t need =
      p.n_slot > 1 ? static_cast<size_t>(R) * p.n_slot * sizeof(State) : 0;
  if (workspace_bytes < need || (need && !workspace)) return WEDLM_E_WORKSPACE;
  LmArgs a{};
  a.hidden = hidden; a.w = w_vocab; a.R = R; a.Hd = Hd; a.V = V;
  a.n_rg = p.n_rg; a.n_slot = p.n_slot; a.nblk = p.nblk;
  a.c2 = 1.4426950408889634074 / temperature;
  a.argmax = argmax; a.entropy = entropy; a.pmax = pmax;
  a.ws = static_cast<State*>(workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  // slot = (blockIdx / 8 / n_rg) * 8 + blockIdx % 8: a multiple of 8 per
  // row group covers every slot
  const int64_t grid = 8ll * p.n_rg * ((p.n_slot + 7) / 8);
  if (grid > (1ll << 30)) return WEDLM_E_SHAPE;
  if (p.ks_spw > 0) {
    const dim3 g(p.n_slot), b(kKsWaves * kWave);
    if (p.ks_spw == 4)
      hipLaunchKernelGGL((lm_head_ks_kernel<4, kKsPF>), g, b, 0, st, a);
    else
      hipLaunchKernelGGL((lm_head_ks_kernel<8, kKsPF>), g, b, 0, st, a);
    WEDLM_LAUNCH_CHECK();
  } else {
    const bool nt = p.n_rg == 1;
    switch (shape_index(p.sh)) {
      case 0: launch<1, 1, kPF>(nt, grid, st, a); break;
      case 1: launch<2, 1, kPF>(nt, grid, st, a); break;
      case 2: launch<3, 1, 2>(nt, grid, st, a); break;
      case 3: launch<2, 2, 2, 2>(nt, grid, st, a); break;
      case 4: launch<2, 4, 2, 2>(nt, grid, st, a); break;
      case 5: launch<3, 4, 1, 2>(nt, grid, st, a); break;
      default: launch_dma<4, 4, 2>(nt, grid, st, a); break;
    }
    WEDLM_LAUNCH_CHECK();
  }
  if (p.n_slot > 1) {
    hipLaunchKernelGGL(lm_head_merge_kernel, dim3(R), dim3(kWave), 0, st, a);
    WEDLM_LAUNCH_CHECK();
  }
  return WEDLM_OK;
}
