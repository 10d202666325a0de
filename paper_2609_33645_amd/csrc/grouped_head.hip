// Grouped logits for a stock CTC (Sec. 3.2, Eq. grouped; Prop. 1; Eq. offsupport).
//
// Forward: R[m] = [Z[m, U_0], ..., Z[m, U_{K-1}], log sum_{v in O} exp Z[m, v]] where O is the
// complement of the selected set U.  Its log softmax is exported; its normaliser is the full
// lambda, so the first K columns are the selected log-probabilities and the last is log P_O.
// One vocabulary pass computes the complement's log-sum-exp (the normaliser kernels run with
// a bias that is -inf on the selected rows), the selected raw logits are gathered, and a
// per-frame finalize combines the two into lambda and the exported row.
//
// Backward: from dL/d(log softmax R) to the inputs of the recomputed backward.  With
// sigma = sum_j dlogp_j and c = dlogp_K / P_O, the logit gradient is dlogp_j - sigma p_v on
// selected classes and p_v (c - sigma) on the complement, i.e. scatter_U(G) - g p with
// G_j = dlogp_j - c p_{U_j} and g = sigma - c.  Adding kappa * exp(logp) to dlogp (the other
// common convention for a CTC gradient on log-probabilities) leaves G and g unchanged.
#include "pctc_internal.h"

namespace pctc {

namespace {

__device__ __forceinline__ double wave_sum_dbl(double x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// remap[v] = -1; small = {K, 0}
__global__ void grouped_index_init(int32_t* __restrict__ remap, int V, int32_t* __restrict__ small, int K) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v < V) remap[v] = -1;
  if (v == 0) {
    small[0] = K;
    small[1] = 0;
  }
}

// remap[u_ids[j]] = j; small[1] = 1 on an id outside [0, V) or an id given twice.
__global__ void grouped_index_scatter(const int32_t* __restrict__ u_ids, int K, int V, int32_t* __restrict__ remap,
                                      int32_t* __restrict__ small) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= K) return;
  const int v = u_ids[j];
  if (v < 0 || v >= V) {
    small[1] = 1;
    return;
  }
  if (atomicCAS(&remap[v], -1, j) != -1) small[1] = 1;
}

// bias of the complement pass: -inf on selected rows, b (or 0) elsewhere
__global__ void grouped_comp_bias(const float* __restrict__ bias, const int32_t* __restrict__ remap, int V,
                                  float* __restrict__ bo) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= V) return;
  bo[v] = (remap[v] >= 0) ? -INFINITY : (bias ? bias[v] : 0.f);
}

__global__ void fill_d(double* __restrict__ x, int n, double val) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) x[i] = val;
}

// One wavefront per frame.  On entry row m of logp (pitch K + 1) holds the raw selected
// logits; lse_o[m] is the complement's log-sum-exp.  lambda = log(exp(lse_U) + exp(lse_O)),
// lse_U with the maximum taken exactly, the exponentials in float on exact differences and
// their sum in double.
__global__ void __launch_bounds__(256)
grouped_finalize_kernel(float* __restrict__ logp, int K, int M, const double* __restrict__ lse_o,
                        double* __restrict__ lam) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= M) return;
  float* row = logp + static_cast<int64_t>(m) * (K + 1);
  float mx = -INFINITY;
  int nan = 0;
  for (int j = lane; j < K; j += 64) {
    const float z = row[j];
    nan |= (z != z);
    mx = fmaxf(mx, z);
  }
  mx = wave_max(mx);
  const bool any_nan = __ballot(nan) != 0;
  double s = 0.0;
  if (mx != -INFINITY)
    for (int j = lane; j < K; j += 64) s += static_cast<double>(fast_exp2((row[j] - mx) * kLog2e));
  s = wave_sum_dbl(s);
  const double lu = (mx == -INFINITY) ? -INFINITY : static_cast<double>(mx) + log(s);
  const double lo = lse_o[m];
  const double hi = fmax(lu, lo);
  double l = (hi == -INFINITY) ? -INFINITY : hi + log1p(exp(fmin(lu, lo) - hi));
  if (any_nan || lo != lo) l = __longlong_as_double(0x7ff8000000000000LL);
  for (int j = lane; j < K; j += 64) row[j] = static_cast<float>(static_cast<double>(row[j]) - l);
  if (lane == 0) {
    row[K] = static_cast<float>(lo - l);
    lam[m] = l;
  }
}

// One wavefront per frame: G[m, j] = dlogp_j - c p_j (pitch K), g[m] = sigma - c.
__global__ void __launch_bounds__(256)
grouped_adapter_kernel(const float* __restrict__ logp, const float* __restrict__ dlogp, int K, int M,
                       float* __restrict__ G, float* __restrict__ g) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= M) return;
  const float* lr = logp + static_cast<int64_t>(m) * (K + 1);
  const float* dr = dlogp + static_cast<int64_t>(m) * (K + 1);
  double sg = 0.0;
  for (int j = lane; j <= K; j += 64) sg += static_cast<double>(dr[j]);
  sg = wave_sum_dbl(sg);
  const double lk = static_cast<double>(lr[K]);
  const double c = (lk > -INFINITY) ? static_cast<double>(dr[K]) / exp(lk) : 0.0;
  float* gr = G + static_cast<int64_t>(m) * K;
  int nz = 0;
  for (int j = lane; j < K; j += 64) {
    const float gj =
        static_cast<float>(static_cast<double>(dr[j]) - c * static_cast<double>(fast_exp2(lr[j] * kLog2e)));
    gr[j] = gj;
    nz |= (gj != 0.f);
  }
  const bool any = __ballot(nz) != 0;
  // The recomputed backward reads g == 0 as a frame that takes no part (true of the lattice's
  // occupancies, where G == 0 then too).  Here g can vanish with G != 0 (e.g. every class
  // selected and a gradient whose rows sum to zero): the smallest normal float keeps the
  // frame, changing its dZ by at most 1.2e-38 p_v.
  float gv = static_cast<float>(sg - c);
  if (gv == 0.f && any) gv = 1.17549435e-38f;
  if (lane == 0) g[m] = gv;
}

}  // namespace

hipError_t launch_grouped_index(const int32_t* u_ids, int K, int V, int32_t* remap, int32_t* small,
                                hipStream_t stream) {
  hipLaunchKernelGGL(grouped_index_init, dim3((V + 255) / 256), dim3(256), 0, stream, remap, V, small, K);
  if (K > 0)
    hipLaunchKernelGGL(grouped_index_scatter, dim3((K + 255) / 256), dim3(256), 0, stream, u_ids, K, V, remap, small);
  return hipGetLastError();
}

hipError_t launch_grouped_comp_bias(const float* bias, const int32_t* remap, int V, float* bo, hipStream_t stream) {
  hipLaunchKernelGGL(grouped_comp_bias, dim3((V + 255) / 256), dim3(256), 0, stream, bias, remap, V, bo);
  return hipGetLastError();
}

hipError_t launch_fill_d(double* x, int n, double val, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_d, dim3((n + 255) / 256), dim3(256), 0, stream, x, n, val);
  return hipGetLastError();
}

hipError_t launch_grouped_finalize(float* logp, int K, int M, const double* lse_o, double* lam, hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  Prof pr("grouped_finalize", stream);
  hipLaunchKernelGGL(grouped_finalize_kernel, dim3((M + 3) / 4), dim3(256), 0, stream, logp, K, M, lse_o, lam);
  return hipGetLastError();
}

hipError_t launch_grouped_adapter(const float* logp, const float* dlogp, int K, int M, float* G, float* g,
                                  hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  Prof pr("grouped_adapter", stream);
  hipLaunchKernelGGL(grouped_adapter_kernel, dim3((M + 3) / 4), dim3(256), 0, stream, logp, dlogp, K, M, G, g);
  return hipGetLastError();
}

}  // namespace pctc
