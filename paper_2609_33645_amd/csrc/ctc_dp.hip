// Alignment lattice of Pruned CTC (Sec. 3.1 CTC; Sec. 3.3 and App. B.3 beam pruning;
// Algorithm 1 lattice, total scores, zeroing of nonfinite losses and dL/dS).
//
// The lattice of utterance n is the extended label sequence l' = (blank, y1, blank, ...,
// yU, blank) of S' = 2U+1 states per frame; it is implicit (states are indices).  Arcs:
// start -> (0, s) for s < 2; (t-1, s) -> (t, s); (t-1, s-1) -> (t, s); (t-1, s-2) -> (t, s)
// when l'_s is a label different from l'_{s-2}; (T-1, s) -> end for s >= S'-2.
//
// Kernels:
//   dp_prep      per utterance: alignability T >= U + r (App. B.1), duplicate-label links,
//                frame -> utterance map.
//   dp_pass      one wavefront per (utterance, direction); lane l holds states
//                [lQ, lQ+Q).  Viterbi (max-plus, float) or total score (log-sum-exp,
//                accumulated in double), renormalised every frame by the wave maximum
//                with the running offsets kept in double.
//   dp_mask      beam rule: keep an arc iff the best complete alignment through it scores
//                at least (best alignment) - beam - slack.
//   dp_occupancy gamma_t(s) = alpha_t(s) beta_t(s) / P, summed per selected class into
//                G = dL/dS = -gamma (Algorithm 1 output), and g = row sums of G.
//   loss_reduce  sum of finite per-utterance losses (Algorithm 1, zero nonfinite).
#include <type_traits>

#include "pctc_internal.h"
#include "prunedctc.h"

namespace pctc {

constexpr float kNeg = -1.0e30f;  // "impossible" score; absorbs finite additions
constexpr int kMaxQ = 32;         // most states per lane of a lattice pass (2U+1 <= 64 kMaxQ)
static_assert(2 * PCTC_MAX_TARGET + 1 <= 64 * kMaxQ, "the longest target fits a lattice pass");
// arc flags of a pass without a mask: every arc kept
constexpr int kAllArcs = 0x0f;
// bytes the mask region extends past its last cell: a pass reads each lane's flags as whole
// aligned words, up to (kMaxQ + 3) / 4 + 1 words from the lane's first cell
constexpr int kMaskPad = 64;
static_assert(4 * ((kMaxQ + 3) / 4 + 1) <= kMaskPad, "mask padding covers a lane's word reads");

DpPlan plan_dp(int N, const int32_t* T, const int32_t* U, float beam) {
  DpPlan p{};
  p.N = N;
  p.pruned = (beam == beam) && beam >= 0.f && beam < INFINITY;
  int64_t M = 0, Y = 0, L = 0;
  int Smax = 1;
  for (int n = 0; n < N; ++n) {
    M += T[n];
    Y += U[n];
    L += static_cast<int64_t>(T[n]) * (2 * U[n] + 1);
    Smax = U[n] * 2 + 1 > Smax ? U[n] * 2 + 1 : Smax;
  }
  p.M = static_cast<int>(M);
  p.Y = static_cast<int>(Y);
  p.Smax = Smax;
  p.lattice = L;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o += align_up(bytes > 0 ? bytes : 1, 256);
    return at;
  };
  p.off_toff = take((N + 1) * sizeof(int32_t));
  p.off_yoff = take((N + 1) * sizeof(int32_t));
  p.off_soff = take((N + 1) * sizeof(int64_t));
  p.off_frame_utt = take(M * sizeof(int32_t));
  p.off_dup_next = take(Y * sizeof(int32_t));
  p.off_dup_first = take(Y * sizeof(int32_t));
  p.off_logp = take(N * sizeof(double));
  p.off_status = take(N * sizeof(int32_t));
  p.off_tab_fa = take(L * sizeof(float));
  p.off_tab_fb = take(L * sizeof(float));
  p.off_sc_fa = take(M * sizeof(double));
  p.off_sc_fb = take(M * sizeof(double));
  p.off_dummy = take(static_cast<size_t>(2 * N) * 64 * kMaxQ * sizeof(float));
  if (p.pruned) {
    p.off_tab_va = take(L * sizeof(float));
    p.off_tab_vb = take(L * sizeof(float));
    p.off_sc_va = take(M * sizeof(double));
    p.off_sc_vb = take(M * sizeof(double));
    p.off_vbest = take(N * sizeof(double));
    p.off_mask = take(L * sizeof(uint8_t) + kMaskPad);  // the passes read whole words past a row's end
  }
  p.total = o;
  return p;
}

// ---------------------------------------------------------------------------------------

__global__ void dp_prep_kernel(const int32_t* __restrict__ toff, const int32_t* __restrict__ yoff,
                               const int32_t* __restrict__ y_rel, int ncols, int32_t* __restrict__ status,
                               int32_t* __restrict__ dup_next, int32_t* __restrict__ dup_first,
                               int32_t* __restrict__ frame_utt, double* __restrict__ loss_n) {
  const int n = blockIdx.x;
  const int t0 = toff[n], T = toff[n + 1] - t0;
  const int y0 = yoff[n], U = yoff[n + 1] - y0;
  // the utterance's targets in LDS (every entry point rejects U > PCTC_MAX_TARGET before
  // any launch): the duplicate search below compares every pair
  __shared__ int y[PCTC_MAX_TARGET];
  __shared__ int reps, badlab;
  if (threadIdx.x == 0) {
    reps = 0;
    badlab = 0;
  }
  for (int i = threadIdx.x; i < U; i += blockDim.x) y[i] = y_rel[y0 + i];
  __syncthreads();
  int myreps = 0;
  for (int i = threadIdx.x; i < U; i += blockDim.x) {
    if (y[i] < 1 || y[i] >= ncols) badlab = 1;  // not a label column of S
    if (i > 0 && y[i] == y[i - 1]) ++myreps;
    int nx = -1;
    for (int j = i + 1; j < U; ++j)
      if (y[j] == y[i]) {
        nx = j;
        break;
      }
    int first = 1;
    for (int j = 0; j < i; ++j)
      if (y[j] == y[i]) {
        first = 0;
        break;
      }
    dup_next[y0 + i] = nx;
    dup_first[y0 + i] = first;
  }
  if (myreps) atomicAdd(&reps, myreps);
  for (int t = threadIdx.x; t < T; t += blockDim.x) frame_utt[t0 + t] = n;
  __syncthreads();
  if (threadIdx.x == 0) {
    // 3: a relabelled target is not a label column; the lattice is not evaluated
    status[n] = badlab ? 3 : ((T >= U + reps) ? 0 : 1);
    loss_n[n] = 0.0;
  }
}

// ---------------------------------------------------------------------------------------

// Cross-lane moves with DPP (VALU, no LDS round trip).
// wave_shr:1 -> lane l receives lane l-1 (lane 0 keeps `old`); wave_shl:1 -> lane l
// receives lane l+1 (lane 63 keeps `old`).
__device__ __forceinline__ int dpp_up_i(int x, int old) { return __builtin_amdgcn_update_dpp(old, x, 0x138, 0xf, 0xf, false); }
__device__ __forceinline__ int dpp_dn_i(int x, int old) { return __builtin_amdgcn_update_dpp(old, x, 0x130, 0xf, 0xf, false); }
__device__ __forceinline__ float lane_up(float x) { return __int_as_float(dpp_up_i(__float_as_int(x), __float_as_int(kNeg))); }
__device__ __forceinline__ float lane_down(float x) { return __int_as_float(dpp_dn_i(__float_as_int(x), __float_as_int(kNeg))); }
__device__ __forceinline__ double lane_up(double x) {
  const long long b = __double_as_longlong(x);
  const long long nb = __double_as_longlong(static_cast<double>(kNeg));
  const int lo = dpp_up_i(static_cast<int>(b), static_cast<int>(nb));
  const int hi = dpp_up_i(static_cast<int>(b >> 32), static_cast<int>(nb >> 32));
  return __longlong_as_double((static_cast<long long>(hi) << 32) | static_cast<unsigned int>(lo));
}
__device__ __forceinline__ double lane_down(double x) {
  const long long b = __double_as_longlong(x);
  const long long nb = __double_as_longlong(static_cast<double>(kNeg));
  const int lo = dpp_dn_i(static_cast<int>(b), static_cast<int>(nb));
  const int hi = dpp_dn_i(static_cast<int>(b >> 32), static_cast<int>(nb >> 32));
  return __longlong_as_double((static_cast<long long>(hi) << 32) | static_cast<unsigned int>(lo));
}
__device__ __forceinline__ int lane_down_i(int x) { return dpp_dn_i(x, 0); }

// Maximum over the wavefront: DPP reductions within each row of 16 lanes, then the four
// row results read as scalars.
template <int CTRL>
__device__ __forceinline__ float dpp_max_step(float v) {
  return fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, 0xf, 0xf,
                                                               false)));
}
__device__ __forceinline__ float wave_max_dpp(float x) {
  x = dpp_max_step<0xB1>(x);   // quad_perm [1,0,3,2]
  x = dpp_max_step<0x4E>(x);   // quad_perm [2,3,0,1]
  x = dpp_max_step<0x141>(x);  // row_half_mirror
  x = dpp_max_step<0x140>(x);  // row_mirror
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return fmaxf(fmaxf(a, b), fmaxf(c, d));
}

// Max (Viterbi) or log-sum-exp (natural log) of three scores.  The log-sum-exp keeps
// the scores in Acc (double for the total-score pass) and evaluates exp/log in float on
// differences from the maximum, where float is accurate.
template <bool VIT, typename Acc>
__device__ __forceinline__ Acc comb3(Acc a, Acc b, Acc c) {
  const Acc m = fmax(fmax(a, b), c);
  if constexpr (VIT) {
    return m;
  } else {
    const float s = fast_exp2(static_cast<float>(a - m) * kLog2e) + fast_exp2(static_cast<float>(b - m) * kLog2e) +
                    fast_exp2(static_cast<float>(c - m) * kLog2e);
    return m + static_cast<Acc>(fast_log2(s) * kLn2);
  }
}

// Frames of emissions (and arc flags) loaded ahead of the recursion: the frames in flight are
// bounded by the wave's memory counter (63 instructions: per frame Q emission loads, Q table
// stores and the offset store, and with a mask (Q + 3) / 4 + 1 flag-word loads) and by
// registers.
template <int Q, bool MASK>
constexpr int prefetch_depth() {
  return Q <= 4 ? 8 : (Q <= 8 ? 5 : (Q <= 13 ? 3 : 2));
}
// The discarded-mass pass loads one flag byte per state.
template <int Q>
constexpr int prefetch_depth_bytes() {
  return Q <= 3 ? 8 : (Q <= 4 ? 6 : (Q <= 6 ? 4 : (Q <= 8 ? 3 : 2)));
}

// One wavefront per (utterance, direction), natural-log units.  VIT: Viterbi (max-plus)
// accumulated in float; otherwise the total score (log-sum-exp) accumulated in double,
// so the per-frame additions do not round at the magnitude of the emission scores.
// Tables hold scores minus a per-frame offset (rounded to float once); the offsets are
// kept per frame in double.  Emissions and arc flags for the next PF frames are held in
// a register ring so that the gathers are issued well before they are needed.
// kPassWaves wavefronts per workgroup (independent; no barriers), so that the few
// wavefronts of this latency-bound stage occupy few compute units.
constexpr int kPassWaves = 4;

template <int Q, bool VIT, bool MASK>
__global__ void __launch_bounds__(64 * kPassWaves)
dp_pass_kernel(const float* __restrict__ S, int ldS, const int32_t* __restrict__ toff,
               const int32_t* __restrict__ yoff, const int64_t* __restrict__ soff, const int32_t* __restrict__ y_rel,
               int32_t* __restrict__ status, const uint8_t* __restrict__ mask, float* __restrict__ tab_f,
               float* __restrict__ tab_b, double* __restrict__ sc_f, double* __restrict__ sc_b,
               double* __restrict__ total_out, double* __restrict__ loss_n, int N, float* __restrict__ dummy) {
  using Acc = typename std::conditional<VIT, float, double>::type;
  constexpr int PF = prefetch_depth<Q, MASK>();
  const int unit = blockIdx.x * kPassWaves + (threadIdx.x >> 6);  // (utterance, direction)
  if (unit >= 2 * N) return;
  const int n = unit >> 1;
  const int dir = unit & 1;
  const int lane = threadIdx.x & 63;
  if (status[n] != 0) return;
  const int t0 = toff[n], T = toff[n + 1] - t0;
  const int y0 = yoff[n], U = yoff[n + 1] - y0;
  const int Sp = 2 * U + 1;
  const int64_t base = soff[n];
  const int* y = y_rel + y0;
  const Acc neg = kNeg;

  // The blank column index is an opaque per-lane zero: with a literal 0 the compiler would
  // turn the (uniform) blank emission load into a scalar load and wait for it on the spot,
  // defeating the prefetch ring.
  int zero_v;
  asm volatile("v_mov_b32 %0, 0" : "=v"(zero_v));
  int col[Q];
  bool valid[Q], skip_in[Q], skip_out[Q], fin[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int s = lane * Q + q;
    valid[q] = s < Sp;
    col[q] = (valid[q] && (s & 1)) ? y[(s - 1) >> 1] : zero_v;
    skip_in[q] = valid[q] && (s & 1) && s >= 3 && y[(s - 1) >> 1] != y[(s - 3) >> 1];
    const int s2 = s + 2;
    skip_out[q] = (s2 < Sp) && (s2 & 1) && y[(s2 - 1) >> 1] != y[(s2 - 3) >> 1];
    fin[q] = valid[q] && s >= Sp - 2;
  }
  // One frame of emissions and arc flags for this lane's states.  No load, store or prefetch
  // of the frame loop sits under a branch (addresses are clamped in bounds, lanes past the
  // last state store to this wave's dummy row): a branch around memory operations makes the
  // compiler wait for every outstanding load at the join, which would serialise the ring.
  float* const drow = dummy + static_cast<int64_t>(unit) * (64 * Q) + lane * Q;
  auto fetch = [&](int t, float (&e)[Q], int (&mk)[Q]) {
    const float* row = S + static_cast<int64_t>(t0 + t) * ldS;
#pragma unroll
    for (int q = 0; q < Q; ++q) e[q] = row[col[q]];  // invalid states read the blank column (a valid address)
    if constexpr (MASK) {
      // this lane's Q flag bytes (from its first cell, clamped into the row) as the NWD aligned
      // words that cover them, shifted into place: a few loads instead of Q byte loads (the
      // bytes past the row's end, read only for cells past the last state, are not used)
      constexpr int NWD = (Q + 3) / 4 + 1;
      // (the region starts 256-byte aligned, so the offset's low bits are the address's)
      const int64_t a = base + static_cast<int64_t>(t) * Sp + min(lane * Q, Sp - 1);
      const uint32_t* wp = reinterpret_cast<const uint32_t*>(mask + (a & ~static_cast<int64_t>(3)));
      const uint32_t sh = static_cast<uint32_t>(a & 3);
      uint32_t w[NWD];
#pragma unroll
      for (int j = 0; j < NWD; ++j) w[j] = wp[j];
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const uint32_t d = __builtin_amdgcn_alignbyte(w[(q >> 2) + 1], w[q >> 2], sh);
        mk[q] = valid[q] ? static_cast<int>((d >> (8 * (q & 3))) & 0xffu) : 0;
      }
    } else {
#pragma unroll
      for (int q = 0; q < Q; ++q) mk[q] = valid[q] ? kAllArcs : 0;
    }
  };
  auto renorm_store = [&](Acc (&v)[Q], double& off, float* tab, double* sc, int t) {
    float mx = kNeg;
#pragma unroll
    for (int q = 0; q < Q; ++q) mx = fmaxf(mx, static_cast<float>(v[q]));
    mx = wave_max_dpp(mx);
    if (mx <= kNeg * 0.5f || mx != mx) mx = 0.f;  // all impossible (or NaN): keep as is
#pragma unroll
    for (int q = 0; q < Q; ++q) v[q] = (v[q] <= Acc(kNeg * 0.5f)) ? Acc(kNeg) : v[q] - Acc(mx);
    off += static_cast<double>(mx);
    float* trow = tab + base + static_cast<int64_t>(t) * Sp + lane * Q;
#pragma unroll
    for (int q = 0; q < Q; ++q) *(valid[q] ? trow + q : drow + q) = static_cast<float>(v[q]);
    sc[t0 + t] = off;  // wave-uniform: every lane stores the same value
  };

  float ring_e[PF][Q];
  int ring_m[PF][Q];
  if (dir == 0) {
    // ---------------- forward ----------------
    Acc a[Q];
    {
      float e[Q];
      int mk[Q];
      fetch(0, e, mk);
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const int s = lane * Q + q;
        a[q] = (valid[q] && s < 2 && (mk[q] & 1)) ? static_cast<Acc>(e[q]) : neg;
      }
    }
#pragma unroll
    for (int k = 0; k < PF; ++k) fetch(min(1 + k, T - 1), ring_e[k], ring_m[k]);
    double off = 0.0;
    renorm_store(a, off, tab_f, sc_f, 0);
    // frame t from ring slot k, which then prefetches frame t + PF (clamped to the last)
    auto fstep = [&](int t, float (&re)[Q], int (&rm)[Q]) {
          float e[Q];
          int mk[Q];
#pragma unroll
          for (int q = 0; q < Q; ++q) {
            e[q] = re[q];
            mk[q] = rm[q];
          }
          fetch(min(t + PF, T - 1), re, rm);
          const Acc up1 = lane_up(a[Q - 1]);
          const Acc up2 = (Q >= 2) ? lane_up(a[Q >= 2 ? Q - 2 : 0]) : lane_up(up1);
          Acc na[Q];
#pragma unroll
          for (int q = 0; q < Q; ++q) {
            const Acc p0 = a[q];
            const Acc p1 = (q >= 1) ? a[q >= 1 ? q - 1 : 0] : up1;
            const Acc p2 = (q >= 2) ? a[q >= 2 ? q - 2 : 0] : (q == 1 ? up1 : up2);
            const Acc c0 = (mk[q] & 1) ? p0 : neg;
            const Acc c1 = (mk[q] & 2) ? p1 : neg;
            const Acc c2 = (skip_in[q] && (mk[q] & 4)) ? p2 : neg;
            na[q] = valid[q] ? static_cast<Acc>(e[q]) + comb3<VIT, Acc>(c0, c1, c2) : neg;
          }
#pragma unroll
          for (int q = 0; q < Q; ++q) a[q] = na[q];
          renorm_store(a, off, tab_f, sc_f, t);
    };
    int tb = 1;
    for (; tb + PF <= T; tb += PF) {
#pragma unroll
      for (int k = 0; k < PF; ++k) fstep(tb + k, ring_e[k], ring_m[k]);
    }
#pragma unroll
    for (int k = 0; k < PF; ++k)
      if (tb + k < T) fstep(tb + k, ring_e[k], ring_m[k]);
    // total over final states (with final-arc flags)
    int fk[Q];
    {
      float e[Q];
      fetch(T - 1, e, fk);
    }
    float fm = kNeg;
#pragma unroll
    for (int q = 0; q < Q; ++q)
      if (fin[q] && (fk[q] & 8)) fm = fmaxf(fm, static_cast<float>(a[q]));
    fm = wave_max_dpp(fm);
    double total;
    if (VIT) {
      total = off + static_cast<double>(fm);
    } else {
      float s = 0.f;
#pragma unroll
      for (int q = 0; q < Q; ++q)
        if (fin[q] && (fk[q] & 8)) s += fast_exp2(static_cast<float>(a[q] - Acc(fm)) * kLog2e);
      s = wave_sum(s);
      total = off + static_cast<double>(fm) + static_cast<double>(fast_log2(s) * kLn2);
      if (fm <= kNeg * 0.5f) total = -INFINITY;
    }
    if (lane == 0) {
      total_out[n] = total;
      if (!VIT) {
        const double L = -total;
        const bool finite = (L == L) && L < INFINITY && L > -INFINITY;
        loss_n[n] = finite ? L : 0.0;
        if (!finite) status[n] = 2;
      }
    }
  } else {
    // ---------------- backward ----------------
    Acc b[Q];
    {
      float e[Q];
      int mk[Q];
      fetch(T - 1, e, mk);
#pragma unroll
      for (int q = 0; q < Q; ++q) b[q] = (fin[q] && (mk[q] & 8)) ? Acc(0) : neg;
    }
    // ring slot k holds frame (T-1) - k - ... : frames T-1, T-2, ... are consumed as t+1
#pragma unroll
    for (int k = 0; k < PF; ++k) fetch(max(T - 1 - k, 0), ring_e[k], ring_m[k]);
    double off = 0.0;
    renorm_store(b, off, tab_b, sc_b, T - 1);
    // frame t uses the emissions and arcs of frame t + 1 from ring slot k, which then
    // prefetches frame t + 1 - PF (clamped to the first)
    auto bstep = [&](int t, float (&re)[Q], int (&rm)[Q]) {
          float e[Q];
          int mk[Q];
#pragma unroll
          for (int q = 0; q < Q; ++q) {
            e[q] = re[q];
            mk[q] = rm[q];
          }
          fetch(max(t + 1 - PF, 0), re, rm);
          Acc nb[Q];
#pragma unroll
          for (int q = 0; q < Q; ++q) nb[q] = valid[q] ? static_cast<Acc>(e[q]) + b[q] : neg;
          const Acc dn0 = lane_down(nb[0]);
          const Acc dn1 = (Q >= 2) ? lane_down(nb[Q >= 2 ? 1 : 0]) : lane_down(dn0);
          const int mdn0 = lane_down_i(mk[0]);
          const int mdn1 = (Q >= 2) ? lane_down_i(mk[Q >= 2 ? 1 : 0]) : lane_down_i(mdn0);
          Acc nbb[Q];
#pragma unroll
          for (int q = 0; q < Q; ++q) {
            const Acc s0 = nb[q];
            const Acc s1 = (q + 1 < Q) ? nb[q + 1 < Q ? q + 1 : 0] : dn0;
            const Acc s2 = (q + 2 < Q) ? nb[q + 2 < Q ? q + 2 : 0] : (q + 1 < Q ? dn0 : dn1);
            const int m0 = mk[q];
            const int m1 = (q + 1 < Q) ? mk[q + 1 < Q ? q + 1 : 0] : mdn0;
            const int m2 = (q + 2 < Q) ? mk[q + 2 < Q ? q + 2 : 0] : (q + 1 < Q ? mdn0 : mdn1);
            const Acc c0 = (m0 & 1) ? s0 : neg;
            const Acc c1 = (m1 & 2) ? s1 : neg;
            const Acc c2 = (skip_out[q] && (m2 & 4)) ? s2 : neg;
            nbb[q] = valid[q] ? comb3<VIT, Acc>(c0, c1, c2) : neg;
          }
#pragma unroll
          for (int q = 0; q < Q; ++q) b[q] = nbb[q];
          renorm_store(b, off, tab_b, sc_b, t);
    };
    int tb = T - 2;
    for (; tb - (PF - 1) >= 0; tb -= PF) {
#pragma unroll
      for (int k = 0; k < PF; ++k) bstep(tb - k, ring_e[k], ring_m[k]);
    }
#pragma unroll
    for (int k = 0; k < PF; ++k)
      if (tb - k >= 0) bstep(tb - k, ring_e[k], ring_m[k]);
  }
}

// ---------------------------------------------------------------------------------------

// One workgroup per frame.  Margin of each arc into (t, s):
//   alpha^(t-1, s') + E_t(s) + beta^(t, s) - (best - beam - slack) >= 0 keeps it.
__global__ void dp_mask_kernel(const float* __restrict__ S, int ldS, const int32_t* __restrict__ toff,
                               const int32_t* __restrict__ yoff, const int64_t* __restrict__ soff,
                               const int32_t* __restrict__ y_rel, const int32_t* __restrict__ frame_utt,
                               const int32_t* __restrict__ status, const float* __restrict__ va,
                               const float* __restrict__ vb, const double* __restrict__ sva,
                               const double* __restrict__ svb, const double* __restrict__ vbest, float beam,
                               float slack, uint8_t* __restrict__ mask) {
  const int m = blockIdx.x;
  const int n = frame_utt[m];
  if (status[n] != 0) return;
  const int t0 = toff[n], T = toff[n + 1] - t0;
  const int t = m - t0;
  const int y0 = yoff[n], U = yoff[n + 1] - y0;
  const int Sp = 2 * U + 1;
  const int64_t base = soff[n];
  const int* y = y_rel + y0;
  const double thr = vbest[n] - static_cast<double>(beam) - static_cast<double>(slack);
  const float* row = S + static_cast<int64_t>(m) * ldS;
  // frame offsets: alpha^ at t-1 and beta^ at t
  const float off_arc = (t > 0) ? static_cast<float>(sva[m - 1] + svb[m] - thr) : 0.f;
  const float off_start = static_cast<float>(svb[m] - thr);
  const float off_final = static_cast<float>(sva[m] - thr);
  for (int s = threadIdx.x; s < Sp; s += blockDim.x) {
    const int c = (s & 1) ? y[(s - 1) >> 1] : 0;
    const float e = row[c];
    const float bt = vb[base + static_cast<int64_t>(t) * Sp + s];
    uint8_t bits = 0;
    if (t == 0) {
      if (s < 2 && e + bt + off_start >= 0.f) bits |= 1;
    } else {
      const float* ap = va + base + static_cast<int64_t>(t - 1) * Sp;
      const float through = e + bt + off_arc;
      if (ap[s] + through >= 0.f) bits |= 1;
      if (s >= 1 && ap[s - 1] + through >= 0.f) bits |= 2;
      const bool skip = (s & 1) && s >= 3 && y[(s - 1) >> 1] != y[(s - 3) >> 1];
      if (skip && ap[s - 2] + through >= 0.f) bits |= 4;
    }
    if (t == T - 1 && s >= Sp - 2) {
      const float at = va[base + static_cast<int64_t>(t) * Sp + s];
      if (at + off_final >= 0.f) bits |= 8;
    }
    mask[base + static_cast<int64_t>(t) * Sp + s] = bits;
  }
}

// ---------------------------------------------------------------------------------------

constexpr int kOccFrames = 4;  // frames per block, one wavefront each

// One wavefront per frame (no block barriers: a wavefront's LDS accesses are performed in
// program order, and the fence keeps the compiler from reordering them).
__global__ void __launch_bounds__(64 * kOccFrames)
dp_occupancy_kernel(const int32_t* __restrict__ toff, const int32_t* __restrict__ yoff,
                    const int64_t* __restrict__ soff, const int32_t* __restrict__ y_rel,
                    const int32_t* __restrict__ frame_utt, const int32_t* __restrict__ status,
                    const int32_t* __restrict__ dup_next, const int32_t* __restrict__ dup_first,
                    const float* __restrict__ fa, const float* __restrict__ fb, const double* __restrict__ sfa,
                    const double* __restrict__ sfb, const double* __restrict__ logp,
                    const float* __restrict__ weight, float* __restrict__ G, int ldG, float* __restrict__ g, int M,
                    int Smax) {
  extern __shared__ float gam_all[];  // [kOccFrames][Smax]
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int m = blockIdx.x * kOccFrames + wv;
  if (m >= M) return;
  const int n = frame_utt[m];
  if (status[n] != 0) return;  // G row stays zero, g stays zero
  float* gam = gam_all + wv * Smax;
  const int t0 = toff[n];
  const int t = m - t0;
  const int y0 = yoff[n], U = yoff[n + 1] - y0;
  const int Sp = 2 * U + 1;
  const int64_t rowb = soff[n] + static_cast<int64_t>(t) * Sp;
  const float off = static_cast<float>(sfa[m] + sfb[m] - logp[n]);
  const float w = weight ? weight[n] : 1.f;  // loss weight of the utterance: G = -w gamma
  for (int s = lane; s < Sp; s += 64) {
    const float x = fa[rowb + s] + fb[rowb + s] + off;
    gam[s] = fast_exp2(x * kLog2e);
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
  // blank column: sum over even states (fixed order per lane, then across lanes)
  float bsum = 0.f;
  for (int s = 2 * lane; s < Sp; s += 128) bsum += gam[s];
  // label columns: the first occurrence of each label sums its states in target order
  float lsum = 0.f;
  for (int i = lane; i < U; i += 64) {
    if (!dup_first[y0 + i]) continue;
    float acc = gam[2 * i + 1];
    int j = dup_next[y0 + i];
    while (j >= 0) {
      acc += gam[2 * j + 1];
      j = dup_next[y0 + j];
    }
    G[static_cast<int64_t>(m) * ldG + y_rel[y0 + i]] = -w * acc;
    lsum += acc;
  }
  const float blank_total = wave_sum(bsum);
  const float label_total = wave_sum(lsum);
  if (lane == 0) {
    G[static_cast<int64_t>(m) * ldG + 0] = -w * blank_total;
    g[m] = -w * (blank_total + label_total);
  }
}

// loss = sum over included utterances of w_n L_n (w_n = 1 without weights)
__global__ void loss_reduce_kernel(int N, const double* __restrict__ loss_n, const int32_t* __restrict__ status,
                                   const float* __restrict__ weight, double* __restrict__ loss) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  double s = 0.0;
  for (int n = 0; n < N; ++n)
    if (status[n] == 0) s += (weight ? static_cast<double>(weight[n]) : 1.0) * loss_n[n];
  *loss = s;
}

hipError_t launch_loss_reduce(int N, const double* loss_n, const int32_t* status, const float* weight, double* loss,
                              hipStream_t stream) {
  Prof pr("loss_reduce", stream);
  hipLaunchKernelGGL(loss_reduce_kernel, dim3(1), dim3(64), 0, stream, N, loss_n, status, weight, loss);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Inclusion forecast.  For an included utterance every frame's occupancies sum to one
// (each retained alignment occupies exactly one state per frame), so g_m = -w_n there and
// 0 on excluded utterances.  Before the lattice runs, an utterance is forecast included when
// its targets fit its frames (T_n >= U_n + repeats), w_n != 0 and, when lam is given, every
// frame has a finite normaliser (else a nonfinite normaliser shows up in the lattice's
// status); the lattice's statuses are checked against the forecast afterwards.
// ---------------------------------------------------------------------------------------
__global__ void __launch_bounds__(256)
g_forecast_kernel(const int32_t* __restrict__ toff, const int32_t* __restrict__ yoff, const int32_t* __restrict__ y_rel,
                  const double* __restrict__ lam, const float* __restrict__ weight, float* __restrict__ g_pred,
                  int32_t* __restrict__ pred) {
  const int n = blockIdx.x;
  const int t0 = toff[n], T = toff[n + 1] - t0;
  const int y0 = yoff[n], U = yoff[n + 1] - y0;
  int reps = 0, bad = 0;
  for (int i = 1 + threadIdx.x; i < U; i += blockDim.x) reps += (y_rel[y0 + i] == y_rel[y0 + i - 1]);
  if (lam)
    for (int t = threadIdx.x; t < T; t += blockDim.x) {
      const double l = lam[t0 + t];
      bad |= !(l > -INFINITY && l < INFINITY);  // NaN fails both
    }
  __shared__ int sreps;
  if (threadIdx.x == 0) sreps = 0;
  __syncthreads();
  if (reps) atomicAdd(&sreps, reps);
  const int anybad = __syncthreads_or(bad);
  const float w = weight ? weight[n] : 1.f;
  const bool inc = !anybad && T >= U + sreps && w != 0.f;
  for (int t = threadIdx.x; t < T; t += blockDim.x) g_pred[t0 + t] = inc ? -w : 0.f;
  if (threadIdx.x == 0) pred[n] = inc ? 1 : 0;
}

// flag = 1 if any utterance's inclusion (status 0 and w_n != 0) differs from the forecast
__global__ void forecast_check_kernel(int N, const int32_t* __restrict__ status, const float* __restrict__ weight,
                                      const int32_t* __restrict__ pred, int32_t* __restrict__ flag) {
  int bad = 0;
  for (int n = threadIdx.x; n < N; n += blockDim.x) {
    const float w = weight ? weight[n] : 1.f;
    const int inc = (status[n] == 0 && w != 0.f) ? 1 : 0;
    bad |= (inc != pred[n]);
  }
  bad = __syncthreads_or(bad);
  if (threadIdx.x == 0) flag[0] = bad;
}

hipError_t launch_g_forecast(const DpPlan& plan, void* scratch, const int32_t* y_rel, const double* lam,
                             const float* weight, float* g_pred, int32_t* pred, hipStream_t stream) {
  if (plan.N == 0) return hipSuccess;
  char* sc = static_cast<char*>(scratch);
  const int32_t* toff = reinterpret_cast<const int32_t*>(sc + plan.off_toff);
  const int32_t* yoff = reinterpret_cast<const int32_t*>(sc + plan.off_yoff);
  hipLaunchKernelGGL(g_forecast_kernel, dim3(plan.N), dim3(256), 0, stream, toff, yoff, y_rel, lam, weight, g_pred,
                     pred);
  return hipGetLastError();
}

hipError_t launch_forecast_check(int N, const int32_t* status, const float* weight, const int32_t* pred,
                                 int32_t* flag, hipStream_t stream) {
  hipLaunchKernelGGL(forecast_check_kernel, dim3(1), dim3(256), 0, stream, N, status, weight, pred, flag);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------

template <bool VIT>
static hipError_t launch_pass(int Q, int N, hipStream_t stream, const float* S, int ldS, const int32_t* toff,
                              const int32_t* yoff, const int64_t* soff, const int32_t* y_rel, int32_t* status,
                              const uint8_t* mask, float* tf, float* tb, double* sf, double* sb, double* total,
                              double* loss_n, float* dummy) {
#define PCTC_PASS(QQ)                                                                                         \
  case QQ:                                                                                                    \
    if (mask)                                                                                                 \
      hipLaunchKernelGGL((dp_pass_kernel<QQ, VIT, !VIT>), grid, dim3(64 * kPassWaves), 0, stream, S, ldS, toff, \
                         yoff, soff, y_rel, status, mask, tf, tb, sf, sb, total, loss_n, N, dummy);           \
    else                                                                                                      \
      hipLaunchKernelGGL((dp_pass_kernel<QQ, VIT, false>), grid, dim3(64 * kPassWaves), 0, stream, S, ldS,   \
                         toff, yoff, soff, y_rel, status, nullptr, tf, tb, sf, sb, total, loss_n, N, dummy);  \
    break;
  const dim3 grid((2 * N + kPassWaves - 1) / kPassWaves);
  switch (Q) {
    PCTC_PASS(1)
    PCTC_PASS(2)
    PCTC_PASS(3)
    PCTC_PASS(4)
    PCTC_PASS(6)
    PCTC_PASS(8)
    PCTC_PASS(10)
    PCTC_PASS(13)
    PCTC_PASS(16)
    PCTC_PASS(20)
    PCTC_PASS(24)
    PCTC_PASS(32)
    default:
      return hipErrorInvalidValue;
  }
#undef PCTC_PASS
  return hipGetLastError();
}

static int pick_q(int Smax) {
  static const int qs[] = {1, 2, 3, 4, 6, 8, 10, 13, 16, 20, 24, kMaxQ};
  const int need = (Smax + 63) / 64;
  for (int q : qs)
    if (q >= need) return q;
  return -1;
}

hipError_t launch_ctc_dp(const DpPlan& plan, const int32_t* T, const int32_t* U, const float* S, int ldS,
                         const int32_t* y_rel, float beam, const float* weight, double* loss_n, int32_t* status,
                         float* G, float* g, uint8_t* keep_mask_out, void* scratch, int K_max, hipStream_t stream,
                         void*, int phase) {
  const int N = plan.N;
  const bool prep = phase == kDpAll || phase == kDpFront || phase == kDpPrep;
  const bool vit = phase == kDpAll || phase == kDpFront || phase == kDpVit;
  const bool back = phase == kDpAll || phase == kDpBack;
  char* sc = static_cast<char*>(scratch);
  int32_t* toff = reinterpret_cast<int32_t*>(sc + plan.off_toff);
  int32_t* yoff = reinterpret_cast<int32_t*>(sc + plan.off_yoff);
  int64_t* soff = reinterpret_cast<int64_t*>(sc + plan.off_soff);
  int32_t* frame_utt = reinterpret_cast<int32_t*>(sc + plan.off_frame_utt);
  int32_t* dnext = reinterpret_cast<int32_t*>(sc + plan.off_dup_next);
  int32_t* dfirst = reinterpret_cast<int32_t*>(sc + plan.off_dup_first);
  double* logp = reinterpret_cast<double*>(sc + plan.off_logp);
  float* tfa = reinterpret_cast<float*>(sc + plan.off_tab_fa);
  float* dummy = reinterpret_cast<float*>(sc + plan.off_dummy);
  float* tfb = reinterpret_cast<float*>(sc + plan.off_tab_fb);
  double* sfa = reinterpret_cast<double*>(sc + plan.off_sc_fa);
  double* sfb = reinterpret_cast<double*>(sc + plan.off_sc_fb);
  hipError_t e;
  const int Q = pick_q(plan.Smax);
  if (Q < 0) return hipErrorInvalidValue;
  uint8_t* mask = plan.pruned ? reinterpret_cast<uint8_t*>(sc + plan.off_mask) : nullptr;
  if (prep) {
    // G and g start at zero: excluded utterances and unused columns stay zero.
    if (plan.M > 0) {
      e = hipMemsetAsync(G, 0, static_cast<size_t>(plan.M) * ldS * sizeof(float), stream);
      if (e != hipSuccess) return e;
      e = hipMemsetAsync(g, 0, static_cast<size_t>(plan.M) * sizeof(float), stream);
      if (e != hipSuccess) return e;
    }
    if (N == 0) return hipSuccess;
    {
      Prof pr("dp_prep", stream);
      hipLaunchKernelGGL(dp_prep_kernel, dim3(N), dim3(256), 0, stream, toff, yoff, y_rel, K_max, status, dnext,
                         dfirst, frame_utt, loss_n);
    }
  }
  if (N == 0) return hipGetLastError();
  if (vit) {
    if (plan.pruned) {
      float* tva = reinterpret_cast<float*>(sc + plan.off_tab_va);
      float* tvb = reinterpret_cast<float*>(sc + plan.off_tab_vb);
      double* sva = reinterpret_cast<double*>(sc + plan.off_sc_va);
      double* svb = reinterpret_cast<double*>(sc + plan.off_sc_vb);
      double* vbest = reinterpret_cast<double*>(sc + plan.off_vbest);
      {
        Prof pr("dp_viterbi", stream);
        e = launch_pass<true>(Q, N, stream, S, ldS, toff, yoff, soff, y_rel, status, nullptr, tva, tvb, sva,
                              svb, vbest, loss_n, dummy);
        if (e != hipSuccess) return e;
      }
      if (plan.M > 0) {
        Prof pr("dp_mask", stream);
        hipLaunchKernelGGL(dp_mask_kernel, dim3(plan.M), dim3(256), 0, stream, S, ldS, toff, yoff, soff, y_rel,
                           frame_utt, status, tva, tvb, sva, svb, vbest, beam, kKeepSlack, mask);
      }
    }
  }
  if (!back || N == 0) return hipGetLastError();
  {
    Prof pr("dp_alpha_beta", stream);
    e = launch_pass<false>(Q, N, stream, S, ldS, toff, yoff, soff, y_rel, status, mask, tfa, tfb, sfa, sfb,
                           logp, loss_n, dummy);
    if (e != hipSuccess) return e;
  }
  if (plan.M > 0) {
    Prof pr("dp_occupancy", stream);
    hipLaunchKernelGGL(dp_occupancy_kernel, dim3((plan.M + kOccFrames - 1) / kOccFrames), dim3(64 * kOccFrames),
                       static_cast<size_t>(kOccFrames) * plan.Smax * sizeof(float), stream, toff, yoff, soff, y_rel,
                       frame_utt, status, dnext, dfirst, tfa, tfb, sfa, sfb, logp, weight, G, ldS, g, plan.M,
                       plan.Smax);
  }
  if (keep_mask_out && mask && plan.lattice > 0) {
    e = hipMemcpyAsync(keep_mask_out, mask, plan.lattice, hipMemcpyDeviceToDevice, stream);
    if (e != hipSuccess) return e;
  }
  (void)T;
  (void)U;
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Discarded posterior mass (App. B.3): delta_n = 1 - (sum over retained alignments) /
// (sum over all valid alignments), both of prod_t p_{pi_t}(t) on the same scores.  One
// wavefront per utterance runs the two forward recursions in lockstep in linear space and
// double precision, with one shared scale per frame (the full recursion's maximum), so
// the per-frame scaling cancels in the ratio.  The emission factor exp(S - m_t) (m_t the
// frame's largest selected score) is formed once in float and used by both recursions.
// Utterances that are not alignable get NaN.
// ---------------------------------------------------------------------------------------

// Linear-space neighbour move: lane l receives lane l-1, lane 0 receives 0 (no state).
__device__ __forceinline__ double lane_up_d(double x) {
  const long long b = __double_as_longlong(x);
  const int lo = dpp_up_i(static_cast<int>(b), 0);
  const int hi = dpp_up_i(static_cast<int>(b >> 32), 0);
  return __longlong_as_double((static_cast<long long>(hi) << 32) | static_cast<unsigned int>(lo));
}

__device__ __forceinline__ double wave_max_d(double x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmax(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ double wave_sum_d(double x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

template <int Q>
__global__ void __launch_bounds__(64)
dp_discarded_kernel(const float* __restrict__ S, int ldS, const int32_t* __restrict__ toff,
                    const int32_t* __restrict__ yoff, const int64_t* __restrict__ soff,
                    const int32_t* __restrict__ y_rel, const int32_t* __restrict__ status,
                    const uint8_t* __restrict__ mask, double* __restrict__ delta) {
  const int n = blockIdx.x;
  const int lane = threadIdx.x;
  if (status[n] != 0) {
    if (lane == 0) delta[n] = __longlong_as_double(0x7ff8000000000000LL);
    return;
  }
  const int t0 = toff[n], T = toff[n + 1] - t0;
  const int y0 = yoff[n], U = yoff[n + 1] - y0;
  const int Sp = 2 * U + 1;
  const int64_t base = soff[n];
  const int* y = y_rel + y0;
  int col[Q];
  bool valid[Q], skip_in[Q], fin[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int s = lane * Q + q;
    valid[q] = s < Sp;
    col[q] = (valid[q] && (s & 1)) ? y[(s - 1) >> 1] : 0;
    skip_in[q] = valid[q] && (s & 1) && s >= 3 && y[(s - 1) >> 1] != y[(s - 3) >> 1];
    fin[q] = valid[q] && s >= Sp - 2;
  }
  double af[Q], ap[Q];  // full and retained forward sums, scaled per frame
  // Emissions and arc flags of the next PF frames are held in a register ring; the loop has
  // only loads and no branch around them (clamped addresses), so each frame waits only for
  // its own ring slot.
  constexpr int PF = prefetch_depth_bytes<Q>();
  float ring_e[PF][Q];
  int ring_m[PF][Q];
  auto load_frame = [&](int t, float (&e)[Q], int (&mk)[Q]) {
    const float* row = S + static_cast<int64_t>(t0 + t) * ldS;
    const uint8_t* mrow = mask + base + static_cast<int64_t>(t) * Sp;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const float v = row[col[q]];  // invalid states read the blank column (a valid address)
      e[q] = valid[q] ? v : -INFINITY;
      const int m = static_cast<int>(mrow[min(lane * Q + q, Sp - 1)]);
      mk[q] = valid[q] ? m : 0;
    }
  };
  // exp(e) in double over the whole range without a per-frame shift: 2^x = 2^i 2^(x - i),
  // i = floor(x), the fraction's power in float and the integer one exact
  auto emit = [&](const float (&e)[Q], double (&pe)[Q]) {
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const float x = e[q] * kLog2e;
      const float fi = fminf(fmaxf(floorf(x), -2000.f), 2000.f);
      pe[q] = (valid[q] && x > -INFINITY) ? ldexp(static_cast<double>(fast_exp2(x - fi)), static_cast<int>(fi)) : 0.0;
    }
  };
  // any positive scale serves (both sums take the same one): an approximate reciprocal of
  // the wave maximum
  auto rescale = [&](double (&nf)[Q], double (&np)[Q]) {
    double c = 0.0;
#pragma unroll
    for (int q = 0; q < Q; ++q) c = fmax(c, nf[q]);
    c = wave_max_d(c);
    const double inv = (c > 0.0) ? __builtin_amdgcn_rcp(c) : 0.0;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      af[q] = nf[q] * inv;
      ap[q] = np[q] * inv;
    }
  };
  {  // frame 0: the start arcs
    float e[Q];
    int mk[Q];
    load_frame(0, e, mk);
#pragma unroll
    for (int k = 0; k < PF; ++k) load_frame(min(1 + k, T - 1), ring_e[k], ring_m[k]);
    double pe[Q], nf[Q], np[Q];
    emit(e, pe);
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int s = lane * Q + q;
      nf[q] = (valid[q] && s < 2) ? pe[q] : 0.0;
      np[q] = (valid[q] && s < 2 && (mk[q] & 1)) ? pe[q] : 0.0;
    }
    rescale(nf, np);
  }
  // frame t from ring slot k, which then prefetches frame t + PF (clamped to the last)
  auto step = [&](int t, float (&re)[Q], int (&rm)[Q]) {
    float e[Q];
    int mk[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      e[q] = re[q];
      mk[q] = rm[q];
    }
    load_frame(min(t + PF, T - 1), re, rm);
    double pe[Q], nf[Q], np[Q];
    emit(e, pe);
    const double uf1 = lane_up_d(af[Q - 1]), up1 = lane_up_d(ap[Q - 1]);
    const double uf2 = (Q >= 2) ? lane_up_d(af[Q >= 2 ? Q - 2 : 0]) : lane_up_d(uf1);
    const double up2 = (Q >= 2) ? lane_up_d(ap[Q >= 2 ? Q - 2 : 0]) : lane_up_d(up1);
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const double f0 = af[q], p0 = ap[q];
      const double f1 = (q >= 1) ? af[q >= 1 ? q - 1 : 0] : uf1;
      const double p1 = (q >= 1) ? ap[q >= 1 ? q - 1 : 0] : up1;
      const double f2 = (q >= 2) ? af[q >= 2 ? q - 2 : 0] : (q == 1 ? uf1 : uf2);
      const double p2 = (q >= 2) ? ap[q >= 2 ? q - 2 : 0] : (q == 1 ? up1 : up2);
      nf[q] = valid[q] ? pe[q] * (f0 + f1 + (skip_in[q] ? f2 : 0.0)) : 0.0;
      np[q] = valid[q] ? pe[q] * (((mk[q] & 1) ? p0 : 0.0) + ((mk[q] & 2) ? p1 : 0.0) +
                                  ((skip_in[q] && (mk[q] & 4)) ? p2 : 0.0))
                       : 0.0;
    }
    rescale(nf, np);
  };
  int tb = 1;
  for (; tb + PF <= T; tb += PF) {
#pragma unroll
    for (int k = 0; k < PF; ++k) step(tb + k, ring_e[k], ring_m[k]);
  }
#pragma unroll
  for (int k = 0; k < PF; ++k)
    if (tb + k < T) step(tb + k, ring_e[k], ring_m[k]);
  double sf = 0.0, sp = 0.0;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    if (!fin[q]) continue;
    const int mk = static_cast<int>(mask[base + static_cast<int64_t>(T - 1) * Sp + lane * Q + q]);
    sf += af[q];
    if (mk & 8) sp += ap[q];
  }
  sf = wave_sum_d(sf);
  sp = wave_sum_d(sp);
  if (lane == 0) delta[n] = (sf > 0.0) ? 1.0 - sp / sf : __longlong_as_double(0x7ff8000000000000LL);
}

static hipError_t launch_discarded(int Q, int N, hipStream_t stream, const float* S, int ldS, const int32_t* toff,
                                   const int32_t* yoff, const int64_t* soff, const int32_t* y_rel,
                                   const int32_t* status, const uint8_t* mask, double* delta) {
#define PCTC_DISC(QQ)                                                                                             \
  case QQ:                                                                                                        \
    hipLaunchKernelGGL((dp_discarded_kernel<QQ>), dim3(N), dim3(64), 0, stream, S, ldS, toff, yoff, soff, y_rel, \
                       status, mask, delta);                                                                      \
    break;
  switch (Q) {
    PCTC_DISC(1)
    PCTC_DISC(2)
    PCTC_DISC(3)
    PCTC_DISC(4)
    PCTC_DISC(6)
    PCTC_DISC(8)
    PCTC_DISC(10)
    PCTC_DISC(13)
    PCTC_DISC(16)
    PCTC_DISC(20)
    PCTC_DISC(24)
    PCTC_DISC(32)
    default:
      return hipErrorInvalidValue;
  }
#undef PCTC_DISC
  return hipGetLastError();
}

hipError_t launch_discarded_mass(const DpPlan& plan, const float* S, int ldS, const int32_t* y_rel, const float* beams,
                                 int nbeams, double* delta, void* scratch, int K_max, hipStream_t stream) {
  const int N = plan.N;
  if (N == 0 || nbeams == 0) return hipSuccess;
  if (!plan.pruned) return hipErrorInvalidValue;
  char* sc = static_cast<char*>(scratch);
  int32_t* toff = reinterpret_cast<int32_t*>(sc + plan.off_toff);
  int32_t* yoff = reinterpret_cast<int32_t*>(sc + plan.off_yoff);
  int64_t* soff = reinterpret_cast<int64_t*>(sc + plan.off_soff);
  int32_t* frame_utt = reinterpret_cast<int32_t*>(sc + plan.off_frame_utt);
  int32_t* dnext = reinterpret_cast<int32_t*>(sc + plan.off_dup_next);
  int32_t* dfirst = reinterpret_cast<int32_t*>(sc + plan.off_dup_first);
  int32_t* status = reinterpret_cast<int32_t*>(sc + plan.off_status);
  double* loss_n = reinterpret_cast<double*>(sc + plan.off_logp);  // scratch use only
  float* tva = reinterpret_cast<float*>(sc + plan.off_tab_va);
  float* dummy = reinterpret_cast<float*>(sc + plan.off_dummy);
  float* tvb = reinterpret_cast<float*>(sc + plan.off_tab_vb);
  double* sva = reinterpret_cast<double*>(sc + plan.off_sc_va);
  double* svb = reinterpret_cast<double*>(sc + plan.off_sc_vb);
  double* vbest = reinterpret_cast<double*>(sc + plan.off_vbest);
  uint8_t* mask = reinterpret_cast<uint8_t*>(sc + plan.off_mask);
  {
    Prof pr("dp_prep", stream);
    hipLaunchKernelGGL(dp_prep_kernel, dim3(N), dim3(256), 0, stream, toff, yoff, y_rel, K_max, status, dnext, dfirst,
                       frame_utt, loss_n);
  }
  const int Q = pick_q(plan.Smax);
  if (Q < 0) return hipErrorInvalidValue;
  for (int b = 0; b < nbeams; ++b) {
    hipError_t e;
    {
      Prof pr("dp_viterbi", stream);
      e = launch_pass<true>(Q, N, stream, S, ldS, toff, yoff, soff, y_rel, status, nullptr, tva, tvb, sva, svb,
                            vbest, loss_n, dummy);
      if (e != hipSuccess) return e;
    }
    if (plan.M > 0) {
      Prof pr("dp_mask", stream);
      hipLaunchKernelGGL(dp_mask_kernel, dim3(plan.M), dim3(256), 0, stream, S, ldS, toff, yoff, soff, y_rel, frame_utt,
                         status, tva, tvb, sva, svb, vbest, beams[b], kKeepSlack, mask);
    }
    {
      Prof pr("dp_discarded", stream);
      e = launch_discarded(Q, N, stream, S, ldS, toff, yoff, soff, y_rel, status, mask,
                           delta + static_cast<int64_t>(b) * N);
      if (e != hipSuccess) return e;
    }
  }
  return hipGetLastError();
}

}  // namespace pctc
