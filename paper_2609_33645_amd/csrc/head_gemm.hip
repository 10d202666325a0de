// Vocabulary-head products of Pruned CTC on matrix cores (gfx950).
//
//  * lse_partial: logits tile Z^T = W_tile H_tile^T with a fused online log-sum-exp
//    epilogue over the vocabulary (Eq. lognorm; Algorithm 1 "online log-sum-exp over
//    vocabulary chunks").  The M x V logits are never written; each workgroup keeps a
//    running (max, sum) per frame over its vocabulary partition.
//  * lse_finalize: combines the partitions per frame in double.
//  * gather_s: S = Z[:, U] - lambda for the selected classes, subtraction in double and
//    one rounding to float (Algorithm 1; App. B.1 "Forward computation").
//  * recompute_dz: one vocabulary chunk of dZ = scatter_U(G) - g p, p = exp(Z - lambda),
//    with Z recomputed (Eq. vjp; Algorithm 1 backward loop); stored in the input dtype.
//  * dh_gemm / dw_gemm: dH += dZ W_c and dW_c = dZ^T H (App. A, Step 3).
//
// Every product C[i][j] = sum_k A[i][k] B[j][k] goes through tile_gemm (pctc_device.h).
#include <algorithm>

#include "pctc_internal.h"

namespace pctc {

// Frames (columns) per forward tile, vocabulary rows per forward tile.
constexpr int kFwdBR = 256;
constexpr int kFwdBC = 128;
constexpr int kBwdB = 128;

template <typename T>
struct Cfg;
template <>
struct Cfg<uint16_t> {
  static constexpr int BK = 64;
};
template <>
struct Cfg<float> {
  static constexpr int BK = 32;
};

// blockIdx -> logical work id such that consecutive logical ids land on the same XCD
// (the dispatcher places workgroup b on XCD b % 8).
__device__ __forceinline__ int xcd_swizzle(int bid, int nblocks) {
  const int full = (nblocks / 8) * 8;
  if (bid >= full) return bid;
  return (bid % 8) * (full / 8) + bid / 8;
}

// ---------------------------------------------------------------------------------------
// Forward: online log-sum-exp partials
// ---------------------------------------------------------------------------------------

template <typename T>
__global__ void __launch_bounds__(256)
lse_partial_kernel(const T* __restrict__ H, int M, int D, const T* __restrict__ W, const float* __restrict__ bias,
                   int V, int P, int vper, float2* __restrict__ partials) {
  constexpr int BK = Cfg<T>::BK;
  using Shape = TileShape<T, kFwdBR, kFwdBC, BK>;
  constexpr int FR = Shape::FR, FC = Shape::FC;
  __shared__ __attribute__((aligned(16))) T lds[Shape::kLdsElems];
  const int nMt = (M + kFwdBC - 1) / kFwdBC;
  const int work = xcd_swizzle(blockIdx.x, gridDim.x);
  const int mt = work % nMt;
  const int p = work / nMt;
  const int m0 = mt * kFwdBC;
  const int vbeg = p * vper;
  const int vend = min(V, vbeg + vper);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  Operand<T> A{W, D, V, D, nullptr, nullptr};
  Operand<T> B{H, D, M, D, nullptr, nullptr};
  float run_max[FC], run_sum[FC];
#pragma unroll
  for (int j = 0; j < FC; ++j) {
    run_max[j] = -INFINITY;
    run_sum[j] = 0.f;
  }
  f32x16 acc[FR][FC];
  for (int v0 = vbeg; v0 < vend; v0 += kFwdBR) {
    tile_gemm<T, kFwdBR, kFwdBC, BK, Lay::KMajor, Lay::KMajor>(A, B, v0, m0, 0, D, lds, acc);
    if (bias) {
#pragma unroll
      for (int i = 0; i < FR; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int v = v0 + acc_row<kFwdBR>(wave, lane, i, r);
          const float b = (v < vend) ? bias[v] : 0.f;
#pragma unroll
          for (int j = 0; j < FC; ++j) acc[i][j][r] += b;
        }
    }
    // rows past the partition end take no part in the sums
    if (v0 + kFwdBR > vend) {
#pragma unroll
      for (int i = 0; i < FR; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const bool ok = v0 + acc_row<kFwdBR>(wave, lane, i, r) < vend;
#pragma unroll
          for (int j = 0; j < FC; ++j) acc[i][j][r] = ok ? acc[i][j][r] : -INFINITY;
        }
    }
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      float tmax = -INFINITY;
#pragma unroll
      for (int i = 0; i < FR; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, acc[i][j][r]);
      tmax = fmaxf(tmax, swap_halves(tmax));
      const float nmax = fmaxf(run_max[j], tmax);
      // a column with no finite logit yet (rows masked by a -inf bias) adds nothing
      const float ms = (nmax == -INFINITY) ? 0.f : nmax * kLog2e;
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < FR; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += fast_exp2(fmaf(acc[i][j][r], kLog2e, -ms));
      s += swap_halves(s);
      const float scale = (run_max[j] == -INFINITY) ? 0.f : fast_exp2((run_max[j] - nmax) * kLog2e);
      run_sum[j] = fmaf(run_sum[j], scale, s);
      run_max[j] = nmax;
    }
  }
  // Combine the two wavefronts that share frames (row halves), then write the partial.
  __syncthreads();
  float2* xch = reinterpret_cast<float2*>(lds);  // [2 col halves][FC*32]
  const int rowhalf = wave >> 1, colhalf = wave & 1;
  if (rowhalf == 1 && lane < 32) {
#pragma unroll
    for (int j = 0; j < FC; ++j) xch[colhalf * (FC * 32) + j * 32 + lane] = make_float2(run_max[j], run_sum[j]);
  }
  __syncthreads();
  if (rowhalf == 0 && lane < 32) {
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      const float2 o = xch[colhalf * (FC * 32) + j * 32 + lane];
      const float nmax = fmaxf(run_max[j], o.x);
      float s = 0.f;
      if (run_max[j] != -INFINITY) s += run_sum[j] * fast_exp2((run_max[j] - nmax) * kLog2e);
      if (o.x != -INFINITY) s += o.y * fast_exp2((o.x - nmax) * kLog2e);
      if (nmax != nmax) s = nmax;  // NaN logits propagate
      const int m = m0 + acc_col<kFwdBC>(wave, lane, j);
      if (m < M) partials[static_cast<int64_t>(p) * M + m] = make_float2(nmax, s);
    }
  }
}

// lambda_m from the per-partition (max, sum) pairs: 16 frames per block, 16 lanes per frame
// splitting the partitions; the maximum is exact, the rescaled sum is accumulated in double
// (each term's exponent taken in float on the exact difference to the maximum).  With Zd,
// also S[m][j] = float(Zd[m][j] - lambda_m) for j < *K (one rounding).
constexpr int kFinFrames = 16;
template <int PER>  // partitions per lane held in registers: P <= 16 PER
__global__ void __launch_bounds__(256)
lse_finalize_kernel(const float2* __restrict__ partials, int M, int P, double* __restrict__ lam,
                    float2* __restrict__ lam2, const double* __restrict__ Zd, const int32_t* __restrict__ Kdev,
                    float* __restrict__ S, int ldS, const float* __restrict__ g, float* __restrict__ rowscale,
                    int32_t* __restrict__ einv) {
  const int ph = threadIdx.x & 15;
  const int m = blockIdx.x * kFinFrames + (threadIdx.x >> 4);
  const bool live = m < M;
  // this lane's partitions ph, ph + 16, ... (at most PER), read once
  constexpr int kPer = PER;
  float2 q[kPer];
  float mx = -INFINITY;
  int nan = 0;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int p = ph + 16 * i;
    q[i] = (live && p < P) ? partials[static_cast<int64_t>(p) * M + m] : make_float2(-INFINITY, 0.f);
    nan |= (q[i].x != q[i].x) | (q[i].y != q[i].y);
    mx = fmaxf(mx, q[i].x);
  }
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) {
    mx = fmaxf(mx, __shfl_xor(mx, o, 16));
    nan |= __shfl_xor(nan, o, 16);
  }
  double s = 0.0;
  if (mx != -INFINITY)
#pragma unroll
    for (int i = 0; i < kPer; ++i)
      if (q[i].x != -INFINITY)
        s += static_cast<double>(q[i].y) *
             static_cast<double>(fast_exp2(static_cast<float>(static_cast<double>(q[i].x) - mx) * kLog2e));
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) s += __shfl_xor(s, o, 16);
  if (!live) return;
  double l = static_cast<double>(mx) + log(s);
  if (mx == -INFINITY) l = -INFINITY;
  if (nan) l = __longlong_as_double(0x7ff8000000000000LL);
  if (ph == 0) {
    lam[m] = l;
    const double l2 = l * kLog2eD;
    const float hi = static_cast<float>(l2);
    lam2[m] = make_float2(hi, static_cast<float>(l2 - static_cast<double>(hi)));
    if (g) {
      if (!(l >= kEMin && l <= kEMax)) atomicOr(einv, 1);
      rowscale[m] = static_cast<float>(-static_cast<double>(g[m]) * exp(-l));
    }
  }
  if (Zd) {
    const int K = *Kdev;
    const double* zr = Zd + static_cast<int64_t>(m) * ldS;
    float* sr = S + static_cast<int64_t>(m) * ldS;
#pragma unroll 4
    for (int j = ph; j < K; j += 16) sr[j] = static_cast<float>(zr[j] - l);
  }
}

__global__ void lam2_kernel(const double* __restrict__ lam, int M, float2* __restrict__ lam2) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= M) return;
  const double l2 = lam[m] * kLog2eD;
  const float hi = static_cast<float>(l2);
  lam2[m] = make_float2(hi, static_cast<float>(l2 - static_cast<double>(hi)));
}

int lse_partitions(int M, int V) {
  // Enough workgroups to fill 256 compute units a few times over; the partition count
  // (not V) sets the size of the partial buffer.
  const int nMt = (M + kFwdBC - 1) / kFwdBC;
  int P = (2048 + nMt - 1) / nMt;
  const int vtiles = (V + kFwdBR - 1) / kFwdBR;
  if (P > vtiles) P = vtiles;
  if (P > 256) P = 256;
  if (P < 1) P = 1;
  return P;
}

size_t lse_partial_bytes(int M, int D) {
  return align_up(static_cast<size_t>(lse_max_parts(D)) * M * sizeof(float2), 256);
}

hipError_t launch_lam2(const double* lam, int M, float2* lam2, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  Prof pr("lam2", stream);
  hipLaunchKernelGGL(lam2_kernel, dim3((M + 255) / 256), dim3(256), 0, stream, lam, M, lam2);
  return hipGetLastError();
}

hipError_t launch_lse(int dtype, const void* H, int M, int D, const void* W, const float* bias, int V,
                      float2* partials, double* lam, float2* lam2, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  const int P = lse_partitions(M, V);
  const int vtiles = (V + kFwdBR - 1) / kFwdBR;
  const int vper = ((vtiles + P - 1) / P) * kFwdBR;
  const int Peff = (V + vper - 1) / vper;
  const int nMt = (M + kFwdBC - 1) / kFwdBC;
  int Pfin = Peff;
  if (dtype == 1) {
    hipError_t e1 = launch_lse_partial_bf16(static_cast<const uint16_t*>(H), M, D, static_cast<const uint16_t*>(W), bias,
                                            V, partials, &Pfin, stream);
    if (e1 != hipSuccess) return e1;
  } else {
    Prof pr("lse_partial", stream);
    hipLaunchKernelGGL(lse_partial_kernel<float>, dim3(nMt * Peff), dim3(256), 0, stream,
                       static_cast<const float*>(H), M, D, static_cast<const float*>(W), bias, V, Peff, vper, partials);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_lse_finalize(partials, M, Pfin, lam, lam2, nullptr, nullptr, nullptr, 0, stream);
}

hipError_t launch_lse_partials(int dtype, const void* H, int M, int D, const void* W, const float* bias, int V,
                               float2* partials, int* P_out, hipStream_t stream) {
  *P_out = 0;
  if (M <= 0) return hipSuccess;
  if (dtype == 1)
    return launch_lse_partial_bf16(static_cast<const uint16_t*>(H), M, D, static_cast<const uint16_t*>(W), bias, V,
                                   partials, P_out, stream);
  const int P = lse_partitions(M, V);
  const int vtiles = (V + kFwdBR - 1) / kFwdBR;
  const int vper = ((vtiles + P - 1) / P) * kFwdBR;
  const int Peff = (V + vper - 1) / vper;
  const int nMt = (M + kFwdBC - 1) / kFwdBC;
  *P_out = Peff;
  Prof pr("lse_partial", stream);
  hipLaunchKernelGGL(lse_partial_kernel<float>, dim3(nMt * Peff), dim3(256), 0, stream, static_cast<const float*>(H), M,
                     D, static_cast<const float*>(W), bias, V, Peff, vper, partials);
  return hipGetLastError();
}

hipError_t launch_lse_finalize(const float2* partials, int M, int P, double* lam, float2* lam2, const double* Zd,
                               const int32_t* K, float* S, int ldS, hipStream_t stream, const float* g,
                               float* rowscale, int32_t* einv) {
  if (M <= 0) return hipSuccess;
  if (P < 1 || P > kMaxLseParts) return hipErrorInvalidValue;
  Prof pr("lse_finalize", stream);
  const dim3 grid((M + kFinFrames - 1) / kFinFrames);
  if (P <= 256)
    hipLaunchKernelGGL(lse_finalize_kernel<16>, grid, dim3(256), 0, stream, partials, M, P, lam, lam2, Zd, K, S, ldS,
                       g, rowscale, einv);
  else
    hipLaunchKernelGGL(lse_finalize_kernel<kMaxLseParts / 16>, grid, dim3(256), 0, stream, partials, M, P, lam, lam2,
                       Zd, K, S, ldS, g, rowscale, einv);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Greedy emission head (framewise argmax over V, smallest class id on ties) and the CTC
// collapse of each utterance's argmax sequence (Sec. 3.1: merge repeats, drop blanks)
// ---------------------------------------------------------------------------------------

__device__ __forceinline__ void amax_merge_g(float& bv, int& bi, float ov, int oi) {
  if (ov > bv || (ov == bv && oi < bi)) {
    bv = ov;
    bi = oi;
  }
}

template <typename T>
__global__ void __launch_bounds__(256)
amax_partial_kernel(const T* __restrict__ H, int M, int D, const T* __restrict__ W, const float* __restrict__ bias,
                    int V, int P, int vper, float2* __restrict__ partials) {
  constexpr int BK = Cfg<T>::BK;
  using Shape = TileShape<T, kFwdBR, kFwdBC, BK>;
  constexpr int FR = Shape::FR, FC = Shape::FC;
  __shared__ __attribute__((aligned(16))) T lds[Shape::kLdsElems];
  const int nMt = (M + kFwdBC - 1) / kFwdBC;
  const int work = xcd_swizzle(blockIdx.x, gridDim.x);
  const int mt = work % nMt;
  const int p = work / nMt;
  const int m0 = mt * kFwdBC;
  const int vbeg = p * vper;
  const int vend = min(V, vbeg + vper);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  Operand<T> A{W, D, V, D, nullptr, nullptr};
  Operand<T> B{H, D, M, D, nullptr, nullptr};
  float bv[FC];
  int bi[FC];
#pragma unroll
  for (int j = 0; j < FC; ++j) {
    bv[j] = -INFINITY;
    bi[j] = 0x7fffffff;
  }
  f32x16 acc[FR][FC];
  for (int v0 = vbeg; v0 < vend; v0 += kFwdBR) {
    tile_gemm<T, kFwdBR, kFwdBC, BK, Lay::KMajor, Lay::KMajor>(A, B, v0, m0, 0, D, lds, acc);
#pragma unroll
    for (int j = 0; j < FC; ++j)
#pragma unroll
      for (int i = 0; i < FR; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int v = v0 + acc_row<kFwdBR>(wave, lane, i, r);
          if (v >= vend) continue;
          const float x = acc[i][j][r] + (bias ? bias[v] : 0.f);
          if (x > bv[j]) {
            bv[j] = x;
            bi[j] = v;
          }
        }
  }
#pragma unroll
  for (int j = 0; j < FC; ++j) amax_merge_g(bv[j], bi[j], swap_halves(bv[j]), __shfl_xor(bi[j], 32, 64));
  __syncthreads();
  float2* xch = reinterpret_cast<float2*>(lds);
  const int rowhalf = wave >> 1, colhalf = wave & 1;
  if (rowhalf == 1 && lane < 32) {
#pragma unroll
    for (int j = 0; j < FC; ++j) xch[colhalf * (FC * 32) + j * 32 + lane] = make_float2(bv[j], __int_as_float(bi[j]));
  }
  __syncthreads();
  if (rowhalf == 0 && lane < 32) {
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      const float2 o = xch[colhalf * (FC * 32) + j * 32 + lane];
      amax_merge_g(bv[j], bi[j], o.x, __float_as_int(o.y));
      const int m = m0 + acc_col<kFwdBC>(wave, lane, j);
      if (m < M) partials[static_cast<int64_t>(p) * M + m] = make_float2(bv[j], __int_as_float(bi[j]));
    }
  }
}

// ids[m]: the best of the partitions' (value, id) pairs, in partition order.
// 16 frames per block, 16 lanes per frame splitting the partitions; the merge (larger value,
// then smaller id) is order-independent, so the result does not depend on the split.
__global__ void __launch_bounds__(256)
amax_finalize_kernel(const float2* __restrict__ partials, int M, int P, int32_t* __restrict__ ids) {
  const int ph = threadIdx.x & 15;
  const int m = blockIdx.x * kFinFrames + (threadIdx.x >> 4);
  const bool live = m < M;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  if (live) {
#pragma unroll 4
    for (int p = ph; p < P; p += 16) {
      const float2 q = partials[static_cast<int64_t>(p) * M + m];
      amax_merge_g(bv, bi, q.x, __float_as_int(q.y));
    }
  }
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) {
    const float ov = __shfl_xor(bv, o, 16);
    const int oi = __shfl_xor(bi, o, 16);
    amax_merge_g(bv, bi, ov, oi);
  }
  if (live && ph == 0) ids[m] = (bi == 0x7fffffff) ? 0 : bi;
}

// One wavefront per utterance: frame m keeps its id when it is not blank and differs from
// the previous frame's (Sec. 3.1), and a ballot prefix count gives its output position.
__global__ void __launch_bounds__(256)
ctc_collapse_kernel(const int32_t* __restrict__ ids, const int32_t* __restrict__ toff, int N, int blank,
                    int32_t* __restrict__ tokens, int32_t* __restrict__ lengths) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const int t0 = toff[n], t1 = toff[n + 1];
  int k = 0;
  for (int b = t0; b < t1; b += 64) {
    const int m = b + lane;
    const int c = (m < t1) ? ids[m] : blank;
    const int prev = (m > t0 && m < t1) ? ids[m - 1] : -1;
    const bool keep = c != blank && c != prev;
    const uint64_t mask = __ballot(keep);
    const int before = __popcll(mask & ((uint64_t{1} << lane) - 1));
    if (keep) tokens[t0 + k + before] = c;
    k += __popcll(mask);
  }
  if (lane == 0) lengths[n] = k;
}

hipError_t launch_greedy(int dtype, const void* H, int M, int D, const void* W, const float* bias, int V,
                         const int32_t* toff, int N, int blank, float2* partials, int32_t* ids, int32_t* tokens,
                         int32_t* lengths, hipStream_t stream) {
  if (M > 0) {
    int Pfin;
    if (dtype == 1) {
      hipError_t e = launch_amax_partial_bf16(static_cast<const uint16_t*>(H), M, D, static_cast<const uint16_t*>(W),
                                              bias, V, partials, &Pfin, stream);
      if (e != hipSuccess) return e;
    } else {
      const int P = lse_partitions(M, V);
      const int vtiles = (V + kFwdBR - 1) / kFwdBR;
      const int vper = ((vtiles + P - 1) / P) * kFwdBR;
      Pfin = (V + vper - 1) / vper;
      const int nMt = (M + kFwdBC - 1) / kFwdBC;
      Prof pr("amax_partial", stream);
      hipLaunchKernelGGL(amax_partial_kernel<float>, dim3(nMt * Pfin), dim3(256), 0, stream,
                         static_cast<const float*>(H), M, D, static_cast<const float*>(W), bias, V, Pfin, vper,
                         partials);
    }
    Prof pr("amax_finalize", stream);
    hipLaunchKernelGGL(amax_finalize_kernel, dim3((M + kFinFrames - 1) / kFinFrames), dim3(256), 0, stream, partials,
                       M, Pfin, ids);
  }
  if (N > 0) {
    Prof pr("ctc_collapse", stream);
    hipLaunchKernelGGL(ctc_collapse_kernel, dim3((N + 3) / 4), dim3(256), 0, stream, ids, toff, N, blank, tokens,
                       lengths);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Selected-class log-probabilities S
// ---------------------------------------------------------------------------------------

template <typename T>
__global__ void __launch_bounds__(256, 2)
gather_s_kernel(const T* __restrict__ H, int M, int D, const T* __restrict__ W, const float* __restrict__ bias,
                const int32_t* __restrict__ u_ids, const int32_t* __restrict__ Kdev, int K_max,
                const double* __restrict__ lam, float* __restrict__ S, int ldS) {
  constexpr int BK = Cfg<T>::BK;
  using Shape = TileShape<T, kFwdBR, kFwdBC, BK>;
  constexpr int FR = Shape::FR, FC = Shape::FC;
  __shared__ __attribute__((aligned(16))) T lds[Shape::kLdsElems];
  const int nMt = (M + kFwdBC - 1) / kFwdBC;
  const int mt = blockIdx.x % nMt;
  const int jt = blockIdx.x / nMt;
  const int K = *Kdev;
  const int j0 = jt * kFwdBR;
  if (j0 >= K) return;
  const int m0 = mt * kFwdBC;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  Operand<T> A{W, D, K_max, D, u_ids, Kdev};
  Operand<T> B{H, D, M, D, nullptr, nullptr};
  f32x16 acc[FR][FC];
  tile_gemm<T, kFwdBR, kFwdBC, BK, Lay::Gathered, Lay::KMajor>(A, B, j0, m0, 0, D, lds, acc);
#pragma unroll
  for (int j = 0; j < FC; ++j) {
    const int m = m0 + acc_col<kFwdBC>(wave, lane, j);
    if (m >= M) continue;
    const double l = lam[m];
#pragma unroll
    for (int i = 0; i < FR; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int jj = j0 + acc_row<kFwdBR>(wave, lane, i, r);
        if (jj < K) {
          double z = static_cast<double>(acc[i][j][r]);
          if (bias) z += static_cast<double>(bias[u_ids[jj]]);
          S[static_cast<int64_t>(m) * ldS + jj] = static_cast<float>(z - l);
        }
      }
  }
}

hipError_t launch_gather_s(int dtype, const void* H, int M, int D, const void* W, const float* bias,
                           const int32_t* u_ids, const int32_t* K, int K_max, const double* lam, float* S, int ldS,
                           hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  if (dtype == 1)
    return launch_gather_s_bf16(static_cast<const uint16_t*>(H), M, D, static_cast<const uint16_t*>(W), bias, u_ids, K,
                                K_max, lam, S, ldS, stream);
  const int nMt = (M + kFwdBC - 1) / kFwdBC;
  const int nJt = (K_max + kFwdBR - 1) / kFwdBR;
  Prof pr("gather_s", stream);
  hipLaunchKernelGGL(gather_s_kernel<float>, dim3(nMt * nJt), dim3(256), 0, stream, static_cast<const float*>(H), M, D,
                     static_cast<const float*>(W), bias, u_ids, K, K_max, lam, S, ldS);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Backward
// ---------------------------------------------------------------------------------------

template <typename T>
__device__ __forceinline__ T to_elem(float x);
template <>
__device__ __forceinline__ uint16_t to_elem<uint16_t>(float x) {
  return f32_to_bf16(x);
}
template <>
__device__ __forceinline__ float to_elem<float>(float x) {
  return x;
}

// dZ chunk [M][chunk] (row pitch `chunk`): columns v_local in [0, cw) hold
// scatter_U(G) - g p for vocabulary id c0 + v_local; columns in [cw, tile end) hold 0.
template <typename T>
__global__ void __launch_bounds__(256, 2)
recompute_dz_kernel(const T* __restrict__ H, int M, int D, const T* __restrict__ W, const float* __restrict__ bias,
                    int c0, int cw, const float2* __restrict__ lam2, const float* __restrict__ G, int ldG,
                    const float* __restrict__ g, const int32_t* __restrict__ remap, T* __restrict__ dZ, int chunk) {
  constexpr int BK = Cfg<T>::BK;
  using Shape = TileShape<T, kFwdBR, kFwdBC, BK>;
  constexpr int FR = Shape::FR, FC = Shape::FC;
  __shared__ __attribute__((aligned(16))) T lds[Shape::kLdsElems];
  __shared__ int sel[kFwdBR];
  const int nMt = (M + kFwdBC - 1) / kFwdBC;
  const int work = xcd_swizzle(blockIdx.x, gridDim.x);
  const int mt = work % nMt;
  const int vt = work / nMt;
  const int m0 = mt * kFwdBC;
  const int vl0 = vt * kFwdBR;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  {
    const int vl = vl0 + tid;
    sel[tid] = (vl < cw) ? remap[c0 + vl] : -1;
  }
  const int any_sel = __syncthreads_or(sel[tid] >= 0);
  Operand<T> A{W + static_cast<int64_t>(c0) * D, D, cw, D, nullptr, nullptr};
  Operand<T> B{H, D, M, D, nullptr, nullptr};
  f32x16 acc[FR][FC];
  tile_gemm<T, kFwdBR, kFwdBC, BK, Lay::KMajor, Lay::KMajor>(A, B, vl0, m0, 0, D, lds, acc);
#pragma unroll
  for (int j = 0; j < FC; ++j) {
    const int m = m0 + acc_col<kFwdBC>(wave, lane, j);
    if (m >= M) continue;
    const float gm = g[m];
    const float2 l2 = lam2[m];
    const bool inc = (gm != 0.f);
#pragma unroll
    for (int i = 0; i < FR; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int rl0 = acc_row<kFwdBR>(wave, lane, i, 4 * q);  // 4 consecutive rows
        T out[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int rl = rl0 + e;
          const int vl = vl0 + rl;
          float val = 0.f;
          if (inc && vl < cw) {
            const float z = acc[i][j][4 * q + e] + (bias ? bias[c0 + vl] : 0.f);
            const float t = fmaf(z, kLog2e, -l2.x) - l2.y;
            val = -gm * fast_exp2(t);
            if (any_sel) {
              const int jj = sel[rl];
              if (jj >= 0) val += G[static_cast<int64_t>(m) * ldG + jj];
            }
          }
          out[e] = to_elem<T>(val);
        }
        T* dst = dZ + static_cast<int64_t>(m) * chunk + vl0 + rl0;
        if constexpr (sizeof(T) == 2) {
          u32x2 w = {static_cast<uint32_t>(out[0]) | (static_cast<uint32_t>(out[1]) << 16),
                     static_cast<uint32_t>(out[2]) | (static_cast<uint32_t>(out[3]) << 16)};
          *reinterpret_cast<u32x2*>(dst) = w;
        } else {
          *reinterpret_cast<float4*>(dst) = make_float4(out[0], out[1], out[2], out[3]);
        }
      }
  }
}

// part[s][M][D] += dZ[:, slice s] . W[c0 + slice s, :]; the first chunk (c0 == 0) writes
// every slice instead (zeros when its k range is empty), so the partials need no clearing.
template <typename T>
__global__ void __launch_bounds__(256, 2)
dh_gemm_kernel(const T* __restrict__ dZ, int M, int chunk, const T* __restrict__ W, int D, int c0, int cw,
               int slice, float* __restrict__ part) {
  constexpr int BK = Cfg<T>::BK;
  using Shape = TileShape<T, kBwdB, kBwdB, BK>;
  constexpr int FR = Shape::FR, FC = Shape::FC;
  __shared__ __attribute__((aligned(16))) T lds[Shape::kLdsElems];
  const int nMt = (M + kBwdB - 1) / kBwdB;
  const int nDt = (D + kBwdB - 1) / kBwdB;
  const int work = blockIdx.x;
  const int mt = work % nMt;
  const int dt = (work / nMt) % nDt;
  const int s = work / (nMt * nDt);
  const int m0 = mt * kBwdB, d0 = dt * kBwdB;
  const int kb = s * slice;
  const int ke = min(cw, kb + slice);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  Operand<T> A{dZ, chunk, M, cw, nullptr, nullptr};
  Operand<T> B{W + static_cast<int64_t>(c0) * D, D, D, cw, nullptr, nullptr};
  f32x16 acc[FR][FC];
  tile_gemm<T, kBwdB, kBwdB, BK, Lay::KMajor, Lay::RowMajorT>(A, B, m0, d0, kb, ke, lds, acc);
  const bool first = c0 == 0;
  if (kb >= ke && !first) return;
  float* dst = part + static_cast<int64_t>(s) * M * D;
#pragma unroll
  for (int i = 0; i < FR; ++i)
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      const int d = d0 + acc_col<kBwdB>(wave, lane, j);
      if (d >= D) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + acc_row<kBwdB>(wave, lane, i, r);
        if (m < M) {
          float* p = dst + static_cast<int64_t>(m) * D + d;
          *p = first ? acc[i][j][r] : *p + acc[i][j][r];
        }
      }
    }
}

// dW[c0 + v][:] = sum_m dZ[m][v] Ht[:, m]   (Ht: head input transposed, excluded frames zero)
template <typename T>
__global__ void __launch_bounds__(256, 2)
dw_gemm_kernel(const T* __restrict__ dZ, int M, int chunk, const T* __restrict__ Ht, int Mp, int D, int c0, int cw,
               float* __restrict__ dW) {
  constexpr int BK = Cfg<T>::BK;
  using Shape = TileShape<T, kBwdB, kBwdB, BK>;
  constexpr int FR = Shape::FR, FC = Shape::FC;
  __shared__ __attribute__((aligned(16))) T lds[Shape::kLdsElems];
  const int nVt = (cw + kBwdB - 1) / kBwdB;
  const int work = xcd_swizzle(blockIdx.x, gridDim.x);
  const int vt = work % nVt;
  const int dt = work / nVt;
  const int v0 = vt * kBwdB, d0 = dt * kBwdB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  Operand<T> A{dZ, chunk, cw, M, nullptr, nullptr};
  Operand<T> B{Ht, Mp, D, M, nullptr, nullptr};
  f32x16 acc[FR][FC];
  tile_gemm<T, kBwdB, kBwdB, BK, Lay::RowMajorT, Lay::KMajor>(A, B, v0, d0, 0, M, lds, acc);
#pragma unroll
  for (int i = 0; i < FR; ++i)
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      const int d = d0 + acc_col<kBwdB>(wave, lane, j);
      if (d >= D) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int v = v0 + acc_row<kBwdB>(wave, lane, i, r);
        if (v < cw) dW[static_cast<int64_t>(c0 + v) * D + d] = acc[i][j][r];
      }
    }
}

// Ht[d][m] = H[m][d] for frames with g[m] != 0, else 0; m in [M, Mp) zero.
template <typename T>
__global__ void ht_build_kernel(const T* __restrict__ H, int M, int D, const float* __restrict__ g, T* __restrict__ Ht,
                                int Mp) {
  __shared__ T tile[64][65];
  const int m0 = blockIdx.x * 64, d0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;  // 256 threads: 64 x 4
  for (int r = ty; r < 64; r += 4) {
    const int m = m0 + r, d = d0 + tx;
    T v = T(0);
    if (m < M && d < D && g[m] != 0.f) v = H[static_cast<int64_t>(m) * D + d];
    tile[r][tx] = v;
  }
  __syncthreads();
  for (int r = ty; r < 64; r += 4) {
    const int d = d0 + r, m = m0 + tx;
    if (d < D && m < Mp) Ht[static_cast<int64_t>(d) * Mp + m] = tile[tx][r];
  }
}

// dH = sum of the split-K partials (+ extra, the union-column part, when given), in order.
// dH = sum of the split-K partials (+ extra, which may be dH itself: each element is read
// before it is written by the same thread)
__global__ void dh_reduce_kernel(const float* __restrict__ part, int splits, int64_t n, const float* extra,
                                 float* dH) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int k = 0; k < splits; ++k) s += part[k * n + i];
  if (extra) s += extra[i];
  dH[i] = s;
}

BwdPlan plan_bwd(int dtype, int M, int D, int V, int chunk) {
  BwdPlan p{};
  int cap;  // columns the gradient buffer holds (sizes the workspace; independent of V)
  if (chunk > 0) {
    // a step never needs more columns than the vocabulary has (rounded up to whole tiles)
    const int vr = (V > 0 ? V + 255 : 256) / 256 * 256;
    p.chunk = cap = chunk < vr ? chunk : vr;
  } else {
    // default buffer: M x cap in the input dtype, about 512 MiB (at most 65536 columns);
    // V is then cut into as few equal chunks (multiples of 256 columns) as fit in it, so
    // that no launch works on a short remainder
    const size_t es0 = (dtype == 1) ? 2 : 4;
    size_t cmax = (static_cast<size_t>(512) << 20) / (es0 * static_cast<size_t>(M > 0 ? M : 1));
    if (cmax > 65536) cmax = 65536;
    cmax = cmax / 256 * 256;
    if (cmax < 256) cmax = 256;
    const size_t v = static_cast<size_t>(V > 0 ? V : 1);
    const size_t n = (v + cmax - 1) / cmax;
    size_t c = ((v + n - 1) / n + 255) / 256 * 256;
    if (c > cmax) c = cmax;
    if (dtype == 1 && D < kWideD) {
      // narrow bf16 heads: whole normaliser partitions (kEAlign columns), so that the first
      // chunk's dZ rows can come from the normaliser (lse_partial_e_bf16)
      size_t n2 = n, c2 = ((v + n2 - 1) / n2 + kEAlign - 1) / kEAlign * kEAlign;
      while (c2 > cmax && c2 > static_cast<size_t>(kEAlign)) {
        ++n2;
        c2 = ((v + n2 - 1) / n2 + kEAlign - 1) / kEAlign * kEAlign;
      }
      if (c2 <= cmax) c = c2;
    }
    p.chunk = static_cast<int>(c);
    cap = static_cast<int>(cmax);
  }
  const size_t es = (dtype == 1) ? 2 : 4;
  const int tr = (dtype == 1) ? 256 : kBwdB;  // dH tile rows of the kernel used
  const int tc = (dtype == 1) ? 256 : kBwdB;
  const int tiles = ((M + tr - 1) / tr) * ((D + tc - 1) / tc);
  // k-slices of the dH product (one workgroup per CU): when the tiles alone make less than
  // two 256-workgroup waves, at most ~12,800 columns per slice (a launch of a few long
  // workgroups is exposed to any CU that is held up); then the fewest slices whose launch
  // fills its waves to at least 90%, else the fullest; at most 8
  const int maxs = p.chunk / 256 < 8 ? (p.chunk / 256 > 0 ? p.chunk / 256 : 1) : 8;
  int mins = (tiles < 512) ? (p.chunk + 12799) / 12800 : 1;
  if (mins > maxs) mins = maxs;
  if (mins < 1) mins = 1;
  int splits = mins;
  double best = -1.0;
  for (int sp = mins; sp <= maxs; ++sp) {
    const int wgs = tiles * sp;
    const double fill = static_cast<double>(wgs) / (256.0 * ((wgs + 255) / 256));
    if (fill > best + 1e-9) {
      best = fill;
      splits = sp;
    }
    if (fill >= 0.9) break;
  }
  p.splits = splits;
  p.Mp = ((M + 63) / 64) * 64;
  p.dz_bytes = align_up(static_cast<size_t>(M) * cap * es, 256);
  p.ht_bytes = align_up(static_cast<size_t>(D) * p.Mp * es, 256);  // >= M x D (bf16 masked copy of H)
  // bf16 with a single slice: the dH product accumulates in the caller's dH (no partial buffer)
  p.part_bytes = (dtype == 1 && splits == 1) ? 0 : align_up(static_cast<size_t>(splits) * M * D * sizeof(float), 256);
  p.lam2_bytes = align_up(static_cast<size_t>(M) * sizeof(float2), 256);
  // bf16: per 128-frame tile column sums of dZ for db
  p.dbpart_bytes = (dtype == 1) ? align_up(static_cast<size_t>((M + 127) / 128) * cap * sizeof(float), 256) : 0;
  // narrow bf16 heads: the dense recompute reads its frames from Hs transposed (whole k-lines)
  p.hst_bytes = (dtype == 1 && D < kWideD && D % 128 == 0) ? align_up(static_cast<size_t>(D) * p.Mp * 2, 256) : 0;
  p.total = p.dz_bytes + p.ht_bytes + p.part_bytes + p.lam2_bytes + p.dbpart_bytes + p.hst_bytes;
  return p;
}

// db[v] = sum over frames of dZ[m][v] for the chunk's columns v < cw.
template <typename T>
__global__ void dz_colsum_kernel(const T* __restrict__ dZ, int M, int chunk, int cw, float* __restrict__ db) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= cw) return;
  float s = 0.f;
  for (int m = 0; m < M; ++m) s += static_cast<float>(dZ[static_cast<int64_t>(m) * chunk + v]);
  db[v] = s;
}

template <typename T>
static hipError_t head_bwd_t(const T* H, int M, int D, const T* W, const float* bias, int V, const float2* lam2,
                             const float* G, int ldG, const float* g, const int32_t* remap, float* dH, float* dW,
                             float* db, char* scratch, const BwdPlan& plan, hipStream_t stream) {
  T* dZ = reinterpret_cast<T*>(scratch);
  T* Ht = reinterpret_cast<T*>(scratch + plan.dz_bytes);
  float* part = reinterpret_cast<float*>(scratch + plan.dz_bytes + plan.ht_bytes);
  const int chunk = plan.chunk;
  const int nMt = (M + kFwdBC - 1) / kFwdBC;
  if (dW) {
    Prof pr("ht_build", stream);
    hipLaunchKernelGGL(ht_build_kernel<T>, dim3(plan.Mp / 64, (D + 63) / 64), dim3(256), 0, stream, H, M, D, g,
                       Ht, plan.Mp);
  }
  int slice = ((chunk / plan.splits + 63) / 64) * 64;
  // split-K slices any chunk fills: the first chunk (the widest) writes them all
  const int nslices = (min(chunk, V) + slice - 1) / slice;
  for (int c0 = 0; c0 < V; c0 += chunk) {
    const int cw = min(chunk, V - c0);
    const int nVt = (cw + kFwdBR - 1) / kFwdBR;
    {
      Prof pr("recompute_dz", stream);
      hipLaunchKernelGGL(recompute_dz_kernel<T>, dim3(nMt * nVt), dim3(256), 0, stream, H, M, D, W, bias, c0, cw,
                         lam2, G, ldG, g, remap, dZ, chunk);
    }
    if (db) {
      Prof pr("db_colsum", stream);
      hipLaunchKernelGGL(dz_colsum_kernel<T>, dim3((cw + 255) / 256), dim3(256), 0, stream, dZ, M, chunk, cw,
                         db + c0);
    }
    if (dH) {
      const int tiles = ((M + kBwdB - 1) / kBwdB) * ((D + kBwdB - 1) / kBwdB);
      const int ns = (cw + slice - 1) / slice;
      Prof pr("dh_gemm", stream);
      hipLaunchKernelGGL(dh_gemm_kernel<T>, dim3(tiles * ns), dim3(256), 0, stream, dZ, M, chunk, W, D, c0, cw,
                         slice, part);
    }
    if (dW) {
      const int grid = ((cw + kBwdB - 1) / kBwdB) * ((D + kBwdB - 1) / kBwdB);
      Prof pr("dw_gemm", stream);
      hipLaunchKernelGGL(dw_gemm_kernel<T>, dim3(grid), dim3(256), 0, stream, dZ, M, chunk, Ht, plan.Mp, D, c0, cw,
                         dW);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (dH) {
    const int64_t n = static_cast<int64_t>(M) * D;
    Prof pr("dh_reduce", stream);
    hipLaunchKernelGGL(dh_reduce_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, stream, part,
                       nslices, n, nullptr, dH);
  }
  return hipGetLastError();
}

uint16_t* bwd_hs(void* scratch, const BwdPlan& plan) {
  return reinterpret_cast<uint16_t*>(static_cast<char*>(scratch) + plan.dz_bytes);
}

uint16_t* bwd_hst(void* scratch, const BwdPlan& plan) {
  if (plan.hst_bytes == 0) return nullptr;
  return reinterpret_cast<uint16_t*>(static_cast<char*>(scratch) + plan.dz_bytes + plan.ht_bytes + plan.part_bytes +
                                     plan.lam2_bytes + plan.dbpart_bytes);
}

static hipError_t head_bwd_bf16(const uint16_t* H, int M, int D, const uint16_t* W, const float* bias, int V,
                                const float2* lam2, const float* G, int ldG, const float* g, const int32_t* remap,
                                const float* S, int ldS, float* dH, float* dW, float* db, char* scratch,
                                const BwdPlan& plan, hipStream_t stream, const BwdSide* side) {
  uint16_t* dZ = reinterpret_cast<uint16_t*>(scratch);
  uint16_t* Hs = bwd_hs(scratch, plan);
  uint16_t* Hst = bwd_hst(scratch, plan);
  // a single split-K slice accumulates straight into dH: no partials and no reduction
  const bool in_place = plan.part_bytes == 0;
  float* part = in_place ? dH : reinterpret_cast<float*>(scratch + plan.dz_bytes + plan.ht_bytes);
  float* dbpart = reinterpret_cast<float*>(scratch + plan.dz_bytes + plan.ht_bytes + plan.part_bytes + plan.lam2_bytes);
  const int chunk = plan.chunk;
  const bool two = side && side->stream;
  hipError_t e;
  // Hs: H with the rows of excluded frames zeroed (read by the recompute and by dW), and its
  // transpose where the recompute reads that
  if (!(side && side->hs_built)) {
    e = Hst ? launch_ht_build_bf16(H, M, D, g, Hs, Hst, plan.Mp, stream) : launch_hs_build_bf16(H, M, D, g, Hs, stream);
    if (e != hipSuccess) return e;
  }
  const int slice = ((chunk / plan.splits + 63) / 64) * 64;
  // split-K slices any chunk fills: the first chunk (the widest) starts them all from zero
  const int nslices = (min(chunk, V) + slice - 1) / slice;
  const int64_t n = static_cast<int64_t>(M) * D;
  const float* dH_extra = side ? side->dH_extra : nullptr;
  int started = two ? 0 : 2;  // works of the second stream enqueued so far
  const int nwork = two ? side->nwork : 0;
  auto start_side = [&](int upto) -> hipError_t {  // enqueue works [started, upto)
    for (; started < upto && started < nwork; ++started) {
      hipError_t err;
      if ((err = hipEventRecord(side->gate[started], stream)) != hipSuccess) return err;
      if ((err = hipStreamWaitEvent(side->stream, side->gate[started], 0)) != hipSuccess) return err;
      if ((err = side->work[started].fn(side->work[started].ctx)) != hipSuccess) return err;
    }
    return hipSuccess;
  };
  bool front_pending = two && side->front.fn;
  auto start_front = [&]() -> hipError_t {
    if (!front_pending) return hipSuccess;
    front_pending = false;
    hipError_t err;
    if ((err = hipEventRecord(side->front_gate, stream)) != hipSuccess) return err;
    if ((err = hipStreamWaitEvent(side->stream, side->front_gate, 0)) != hipSuccess) return err;
    return side->front.fn(side->front.ctx);
  };
  int ci = 0;  // chunk index
  for (int c0 = 0; c0 < V; c0 += chunk, ++ci) {
    const int cw = min(chunk, V - c0);
    const bool last = c0 + chunk >= V;
    const ChunkE* ce = (c0 == 0 && side) ? side->ce : nullptr;
    // the first chunk (the widest) sets the slices; a narrower later chunk spreads its columns
    // over as many slices (shorter ones), so that its dH launch keeps its workgroups
    const int sl = (c0 == 0) ? slice : std::max(64, ((cw + nslices - 1) / nslices + 63) / 64 * 64);
    if (last && two && dH) {
      // the last chunk's dW product runs beside the final dH reduction (second stream)
      e = launch_bwd_chunk_bf16(Hs, M, D, W, bias, c0, cw, lam2, G, ldG, g, remap, S, ldS, dZ, chunk, part, sl,
                                true, true, false, dW, db, dbpart, stream, nullptr, ce, Hst, plan.Mp);
      if (e != hipSuccess) return e;
      if ((e = start_front()) != hipSuccess) return e;
      if ((e = start_side(nwork)) != hipSuccess) return e;
      if ((e = hipEventRecord(side->dh_done, stream)) != hipSuccess) return e;
      if ((e = hipStreamWaitEvent(side->stream, side->dh_done, 0)) != hipSuccess) return e;
      if (in_place) {
        if (side->after_dh.fn && (e = side->after_dh.fn(side->after_dh.ctx)) != hipSuccess) return e;
      } else {
        Prof pr("dh_reduce", side->stream);
        hipLaunchKernelGGL(dh_reduce_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, side->stream,
                           part, nslices, n, dH_extra, dH);
        if ((e = hipGetLastError()) != hipSuccess) return e;
      }
      if (dW) {
        // the union columns' dW_u rides in this launch's last round once their bf16 G is written
        const DwExtra* udw = side->udw.Z ? &side->udw : nullptr;
        if (udw && (e = hipStreamWaitEvent(stream, udw->ready, 0)) != hipSuccess) return e;
        e = launch_bwd_chunk_bf16(Hs, M, D, W, bias, c0, cw, lam2, G, ldG, g, remap, S, ldS, dZ, chunk, part, sl,
                                  false, false, true, dW, db, dbpart, stream, udw, ce, Hst, plan.Mp);
        if (e != hipSuccess) return e;
      }
    } else if (front_pending) {
      // the first chunk: the second stream's front starts beside its dW product, not its dH
      e = launch_bwd_chunk_bf16(Hs, M, D, W, bias, c0, cw, lam2, G, ldG, g, remap, S, ldS, dZ, chunk, part, sl,
                                true, dH != nullptr, false, dW, db, dbpart, stream, nullptr, ce, Hst, plan.Mp);
      if (e != hipSuccess) return e;
      if ((e = start_front()) != hipSuccess) return e;
      e = launch_bwd_chunk_bf16(Hs, M, D, W, bias, c0, cw, lam2, G, ldG, g, remap, S, ldS, dZ, chunk, part, sl,
                                false, false, dW != nullptr, dW, db, dbpart, stream, nullptr, ce, Hst, plan.Mp);
      if (e != hipSuccess) return e;
      if ((e = start_side(last ? nwork : ci + 1)) != hipSuccess) return e;
    } else {
      e = launch_bwd_chunk_bf16(Hs, M, D, W, bias, c0, cw, lam2, G, ldG, g, remap, S, ldS, dZ, chunk, part, sl,
                                true, dH != nullptr, dW != nullptr, dW, db, dbpart, stream, nullptr, ce, Hst, plan.Mp);
      if (e != hipSuccess) return e;
      if ((e = start_side(last ? nwork : ci + 1)) != hipSuccess) return e;
    }
  }
  if ((e = start_front()) != hipSuccess) return e;
  if ((e = start_side(nwork)) != hipSuccess) return e;
  if (two) {
    // the second stream's work (its union-column part and, with dH, the reduction) is done
    // before this call's work on the caller's stream is
    if ((e = hipEventRecord(side->reduced, side->stream)) != hipSuccess) return e;
    if ((e = hipStreamWaitEvent(stream, side->reduced, 0)) != hipSuccess) return e;
  } else if (dH && !in_place) {
    Prof pr("dh_reduce", stream);
    hipLaunchKernelGGL(dh_reduce_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, stream, part,
                       nslices, n, dH_extra, dH);
  }
  return hipGetLastError();
}

hipError_t launch_head_bwd(int dtype, const void* H, int M, int D, const void* W, const float* bias, int V,
                           const float2* lam2, const float* G, int ldG, const float* g, const int32_t* remap,
                           const float* S, int ldS, float* dH, float* dW, float* db, void* scratch,
                           const BwdPlan& plan, hipStream_t stream, const BwdSide* side) {
  if (M <= 0) {
    if (db) {
      hipError_t e = hipMemsetAsync(db, 0, static_cast<size_t>(V) * sizeof(float), stream);
      if (e != hipSuccess) return e;
    }
    if (dW) return hipMemsetAsync(dW, 0, static_cast<size_t>(V) * D * sizeof(float), stream);
    return hipSuccess;
  }
  char* sc = static_cast<char*>(scratch);
  if (dtype == 1)
    return head_bwd_bf16(static_cast<const uint16_t*>(H), M, D, static_cast<const uint16_t*>(W), bias, V, lam2, G, ldG,
                         g, remap, S, ldS, dH, dW, db, sc, plan, stream, side);
  return head_bwd_t<float>(static_cast<const float*>(H), M, D, static_cast<const float*>(W), bias, V, lam2, G, ldG, g,
                           remap, dH, dW, db, sc, plan, stream);
}

}  // namespace pctc
