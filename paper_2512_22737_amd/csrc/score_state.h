// Online state of the greedy token, entropy and top probability of one
// softmax(logits / T) row (Sec. 5.2, the H_i of Eq. (11)), shared by the
// kernels that score rows: wedlm_score (fp32 logits from memory) and
// wedlm_lm_head_score (logits formed on MFMA).
//
// A state covers a set of logits relative to their maximum m:
//   R = sum over x < m of 2^y,  S = sum over x < m of -y 2^y  (log2 units),
//   y = (x - m) * log2(e) / T, ties = number of logits equal to m,
//   tok = lowest index holding m.
// States merge associatively; then
//   H = ln(1 + R') + S' / (1 + R'),  p_max = 1 / (1 + R'),  R' = R + ties - 1,
// two non-negative terms, so nothing cancels even when H is ~1e-25.
#ifndef WEDLM_SCORE_STATE_H
#define WEDLM_SCORE_STATE_H

#include "common.h"

namespace wedlm {

constexpr double kLn2d = 0.69314718055994530942;

// Partial result over a set of logits, relative to its maximum m:
//   R = sum over x < m of 2^y,  S = sum over x < m of -y 2^y  (log2 units),
//   y = (x - m) * log2(e) / T, ties = number of logits equal to m,
//   tok = lowest index holding m.
// The entropy needs R' = R + ties - 1 (all terms but the argmax); keeping
// the ties as an exact count avoids subtracting the argmax's 1 from a sum.
struct State {
  float m;
  int tok;
  int ties;
  double R, S;
};

__device__ __forceinline__ State empty_state() {
  return State{kNegInf, 0x7fffffff, 0, 0.0, 0.0};
}

// 2^y for y <= 0 given in fp64: v_exp_f32 on the fp32 head, the tail as a
// first-order correction; relative error about one fp32 ulp.  Zero below
// -200 (where the fp32 exponential underflows anyway).  Callers clamp y at
// -256 so that a -inf logit adds 0 (not inf * 0) to S.
__device__ __forceinline__ float exp2_split(double y) {
  const float yh = static_cast<float>(y);
  const float yl = static_cast<float>((y - static_cast<double>(yh)) * kLn2d);
  const float e = __builtin_amdgcn_exp2f(yh);
  return y > -200.0 ? __builtin_fmaf(e, yl, e) : 0.f;
}

// The scale c2 = log2(e)/T: in fp64 for the state arithmetic, and as an
// fp32 head c2h plus tail c2l for the per-logit terms (set once per kernel).
struct ExpScale {
  double c2;
  float c2h, c2l;
};

__device__ __forceinline__ ExpScale exp_scale(double c2) {
  ExpScale sc;
  sc.c2 = c2;
  sc.c2h = static_cast<float>(c2);
  sc.c2l = static_cast<float>(c2 - static_cast<double>(sc.c2h));
  return sc;
}

// Exponent constants of a state whose maximum is m: the split scale, and
// m*c2h as an fp32 head mch plus its exact residual mcl (one fused
// multiply-add), so that no rounding is shared by all the terms of a row.
struct ExpConst {
  float c2h, c2l, m, mch, mcl;
};

__device__ __forceinline__ ExpConst exp_const(float m, const ExpScale& sc) {
  ExpConst k;
  k.c2h = sc.c2h;
  k.c2l = sc.c2l;
  k.m = m;
  k.mch = m * k.c2h;
  k.mcl = __builtin_fmaf(m, k.c2h, -k.mch);
  return k;
}

// One term of the sums: y = (x - m) * c2 in fp32, formed as
// (x*c2h - mch, the product exact inside one fused multiply-add) - mcl
// + (x - m)*c2l, clamped at -256 (a -inf logit, or an empty state's NaN,
// gives 2^-256 = 0: never inf * 0), and 2^y.  What remains are the
// roundings of these few operations, below |y| * 2^-22 relative in 2^y and
// independent from term to term; with y near 0 for the terms that carry a
// row's entropy above 1e-7, that is far inside the 1e-5 relative bar.
__device__ __forceinline__ float exp2_term(float x, const ExpConst& k,
                                           float& y) {
  const float p = __builtin_fmaf(x, k.c2h, -k.mch);
  y = fmaxf(__builtin_fmaf(x - k.m, k.c2l, p - k.mcl), -256.f);
  return __builtin_amdgcn_exp2f(y);   // 0 below about -150
}

// Re-express state st relative to a larger maximum: every old term, the old
// ties included, shifts by dy = (m_old - m_new) * c2 < 0.
__device__ __forceinline__ void shift_state(State& st, float m_new, double c2) {
  if (st.m == kNegInf) { st.R = 0.0; st.S = 0.0; st.ties = 0; return; }
  const double dy = (static_cast<double>(st.m) - m_new) * c2;
  const double all = st.R + st.ties;
  const double e = static_cast<double>(exp2_split(dy));
  st.S = e > 0.0 ? e * (st.S - dy * all) : 0.0;
  st.R = e * all;
  st.ties = 0;
}

// Merge o into st (associative up to rounding; ties keep the lower index).
__device__ __forceinline__ void merge(State& st, State o, double c2) {
  if (o.m == kNegInf) return;
  if (st.m == kNegInf) { st = o; return; }
  if (o.m > st.m) shift_state(st, o.m, c2);
  else if (st.m > o.m) shift_state(o, st.m, c2);
  State r;
  r.m = st.m > o.m ? st.m : o.m;
  r.tok = (st.m == r.m && o.m == r.m) ? min(st.tok, o.tok)
                                      : (st.m == r.m ? st.tok : o.tok);
  r.ties = st.ties + o.ties;
  r.R = st.R + o.R;
  r.S = st.S + o.S;
  st = r;
}

__device__ __forceinline__ State shfl_xor_state(const State& s, int mask) {
  State o;
  o.m = __shfl_xor(s.m, mask);
  o.tok = __shfl_xor(s.tok, mask);
  o.ties = __shfl_xor(s.ties, mask);
  o.R = __shfl_xor(s.R, mask);
  o.S = __shfl_xor(s.S, mask);
  return o;
}

// Add a block of n logits x[k] at indices idx[k] (increasing) to st.  A
// block whose maximum exceeds the running max first raises it (rescaling
// the sums); then every logit adds its term, except those equal to the
// max, which are counted as ties instead (their term is exactly 1 and is
// never summed, so nothing cancels later).
template <int N>
__device__ __forceinline__ void push_block(State& st, const float (&x)[N],
                                           const int (&idx)[N],
                                           const ExpScale& sc) {
  const double c2 = sc.c2;
  float bm = x[0];
#pragma unroll
  for (int k = 1; k < N; ++k) bm = fmaxf(bm, x[k]);
  if (bm > st.m) {
    shift_state(st, bm, c2);
    st.m = bm;
    int t = 0x7fffffff;
#pragma unroll
    for (int k = N - 1; k >= 0; --k) t = (x[k] == bm) ? idx[k] : t;
    st.tok = t;
  }
  const ExpConst kc = exp_const(st.m, sc);
  float r = 0.f, sy = 0.f;
  int ties = 0;
#pragma unroll
  for (int k = 0; k < N; ++k) {
    float yh;
    float e = exp2_term(x[k], kc, yh);
    const bool is_max = x[k] == st.m;
    e = is_max ? 0.f : e;
    ties += is_max ? 1 : 0;
    r += e;
    sy = __builtin_fmaf(-yh, e, sy);
  }
  st.R += r;
  st.S += sy;
  st.ties += ties;
}

__device__ __forceinline__ void finish(const State& st, int64_t idx,
                                       int32_t* argmax, float* entropy,
                                       float* pmax) {
  const double R = st.R + (st.ties - 1);   // every term but the argmax
  const double S = st.S * kLn2d;            // back to nats
  const double H = log1p(R) + S / (1.0 + R);
  argmax[idx] = st.m == kNegInf ? 0 : st.tok;   // an all -inf row: id 0
  entropy[idx] = static_cast<float>(H);
  if (pmax) pmax[idx] = static_cast<float>(1.0 / (1.0 + R));
}


}  // namespace wedlm

#endif  // WEDLM_SCORE_STATE_H
