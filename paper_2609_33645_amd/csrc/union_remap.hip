// Union subset and relabelling (Sec. 3.2 "Reformulation"; Algorithm 1, union/relabel
// steps; App. B.1 "Forward computation").
//
// The selected classes are blank followed by the distinct target labels in increasing id
// order.  One workgroup builds a membership bitmap of the vocabulary in LDS, ranks the set
// bits with a block-wide prefix sum of per-word popcounts, and writes
//   remap[v] = index of v in the union, or -1;   u_ids[j] = j-th selected class;
//   y_rel[i] = remap[targets[i]];                 K = union size.
// Integer work only: the result is exact.
#include "pctc_internal.h"

namespace pctc {

constexpr int kUnionThreads = 1024;

__global__ void __launch_bounds__(kUnionThreads)
union_remap_kernel(const int32_t* __restrict__ targets, int32_t total, int32_t blank, int32_t V,
                   int32_t* __restrict__ remap, int32_t* __restrict__ u_ids, int32_t* __restrict__ y_rel,
                   int32_t* __restrict__ K_out, int32_t* __restrict__ err) {
  extern __shared__ uint32_t lds[];
  const int nwords = (V + 31) >> 5;
  uint32_t* bits = lds;                 // [nwords]
  uint32_t* prefix = lds + nwords;      // [nwords] exclusive rank of the word's first bit
  __shared__ uint32_t scan[kUnionThreads];
  __shared__ int bad;
  const int tid = threadIdx.x;
  if (tid == 0) bad = 0;
  for (int w = tid; w < nwords; w += kUnionThreads) bits[w] = 0u;
  __syncthreads();
  for (int i = tid; i < total; i += kUnionThreads) {
    int v = targets[i];
    if (v < 0 || v >= V || v == blank) {
      bad = 1;
    } else {
      atomicOr(&bits[v >> 5], 1u << (v & 31));
    }
  }
  __syncthreads();
  // Each thread counts a contiguous run of words, then a block scan gives its base rank.
  const int per = (nwords + kUnionThreads - 1) / kUnionThreads;
  const int w0 = tid * per;
  const int w1 = min(nwords, w0 + per);
  uint32_t cnt = 0;
  for (int w = w0; w < w1; ++w) cnt += __popc(bits[w]);
  scan[tid] = cnt;
  __syncthreads();
  for (int off = 1; off < kUnionThreads; off <<= 1) {  // Hillis-Steele inclusive scan
    uint32_t add = (tid >= off) ? scan[tid - off] : 0u;
    __syncthreads();
    scan[tid] += add;
    __syncthreads();
  }
  uint32_t base = scan[tid] - cnt;
  for (int w = w0; w < w1; ++w) {
    prefix[w] = base;
    base += __popc(bits[w]);
  }
  const uint32_t nsel = scan[kUnionThreads - 1];
  __syncthreads();
  for (int v = tid; v < V; v += kUnionThreads) {
    const uint32_t word = bits[v >> 5];
    const uint32_t b = v & 31;
    int r = -1;
    if (v == blank) {
      r = 0;
    } else if ((word >> b) & 1u) {
      r = 1 + static_cast<int>(prefix[v >> 5] + __popc(word & ((1u << b) - 1u)));
      u_ids[r] = v;
    }
    remap[v] = r;
  }
  for (int i = tid; i < total; i += kUnionThreads) {
    int v = targets[i];
    int r = -1;
    if (v >= 0 && v < V && v != blank) {
      const uint32_t word = bits[v >> 5];
      const uint32_t b = v & 31;
      r = 1 + static_cast<int>(prefix[v >> 5] + __popc(word & ((1u << b) - 1u)));
    }
    y_rel[i] = r;
  }
  if (tid == 0) {
    u_ids[0] = blank;
    *K_out = 1 + static_cast<int>(nsel);
    *err = bad;
  }
}

hipError_t launch_union_remap(const int32_t* targets, int32_t total, int32_t blank, int32_t V,
                              int32_t* remap, int32_t* u_ids, int32_t* y_rel, int32_t* K, int32_t* err,
                              hipStream_t stream) {
  const int nwords = (V + 31) >> 5;
  const size_t lds = static_cast<size_t>(2 * nwords) * sizeof(uint32_t);
  Prof p("union_remap", stream);
  hipLaunchKernelGGL(union_remap_kernel, dim3(1), dim3(kUnionThreads), lds, stream, targets, total, blank,
                     V, remap, u_ids, y_rel, K, err);
  return hipGetLastError();
}

// Inverse of a remap table: u_ids[remap[v]] = v and K = 1 + max remap.
__global__ void remap_invert_kernel(const int32_t* __restrict__ remap, int32_t V, int32_t* __restrict__ u_ids,
                                    int32_t* __restrict__ K) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= V) return;
  const int r = remap[v];
  if (r >= 0) {
    u_ids[r] = v;
    atomicMax(K, r + 1);
  }
}

hipError_t launch_remap_invert(const int32_t* remap, int32_t V, int32_t* u_ids, int32_t* K, hipStream_t stream) {
  hipError_t e = hipMemsetAsync(K, 0, sizeof(int32_t), stream);
  if (e != hipSuccess) return e;
  Prof p("remap_invert", stream);
  hipLaunchKernelGGL(remap_invert_kernel, dim3((V + 255) / 256), dim3(256), 0, stream, remap, V, u_ids, K);
  return hipGetLastError();
}

}  // namespace pctc
