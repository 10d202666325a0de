// Union subset and relabelling (Sec. 3.2 "Reformulation"; Algorithm 1, union/relabel
// steps; App. B.1 "Forward computation").
//
// The selected classes are blank followed by the distinct target labels in increasing id
// order.  The vocabulary is cut into blocks of kBlk classes, one workgroup each, in two
// launches:
//   mark:  each block's membership bitmap (every target is read; those in the block set
//          their bit in LDS), stored with the block's member count;
//   rank:  each block's first rank is 1 + the members of all earlier blocks; a prefix over
//          the block's words ranks every member, and the block writes
//            remap[v] = index of v in the union, or -1;   u_ids[j] = j-th selected class;
//            y_rel[i] = remap[targets[i]] for the targets in the block;  K = union size.
// Integer work only: the result is exact.  A workgroup holds 256 bytes of LDS and few
// registers, so these launches run beside the normaliser's products on the same CUs.
#include "pctc_internal.h"

namespace pctc {

constexpr int kBlk = 2048;              // classes per block
constexpr int kBlkWords = kBlk / 32;    // bitmap words per block (one per lane of a wavefront)
constexpr int kUnionThreads = 256;

__global__ void __launch_bounds__(kUnionThreads)
union_mark_kernel(const int32_t* __restrict__ targets, int32_t total, int32_t blank, int32_t V,
                  uint32_t* __restrict__ bits, int32_t* __restrict__ counts, int32_t* __restrict__ err) {
  __shared__ uint32_t word[kBlkWords];
  __shared__ int bad;
  const int tid = threadIdx.x;
  const int lo = blockIdx.x * kBlk, hi = min(V, lo + kBlk);
  if (tid < kBlkWords) word[tid] = 0u;
  if (tid == 0) bad = 0;
  __syncthreads();
  for (int i = tid; i < total; i += kUnionThreads) {
    const int v = targets[i];
    if (v < 0 || v >= V || v == blank) {
      bad = 1;  // a label out of range or equal to blank (every block sees it; block 0 reports)
    } else if (v >= lo && v < hi) {
      atomicOr(&word[(v - lo) >> 5], 1u << (v & 31));
    }
  }
  __syncthreads();
  if (tid < 64) {  // one wavefront: a word per lane, then the block's member count
    const uint32_t w = word[tid];
    bits[static_cast<int64_t>(blockIdx.x) * kBlkWords + tid] = w;
    int c = __popc(w);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) c += __shfl_xor(c, o, 64);
    if (tid == 0) {
      counts[blockIdx.x] = c;
      if (blockIdx.x == 0) *err = bad;
    }
  }
}

__global__ void __launch_bounds__(kUnionThreads)
union_rank_kernel(const int32_t* __restrict__ targets, int32_t total, int32_t blank, int32_t V,
                  const uint32_t* __restrict__ bits, const int32_t* __restrict__ counts, int32_t nblk,
                  int32_t* __restrict__ remap, int32_t* __restrict__ u_ids, int32_t* __restrict__ y_rel,
                  int32_t* __restrict__ K_out) {
  __shared__ uint32_t word[kBlkWords];
  __shared__ int wrank[kBlkWords];   // rank of each word's first member within the block
  __shared__ int part[kUnionThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x;
  const int lo = b * kBlk, hi = min(V, lo + kBlk);
  // members of the earlier blocks (block 0 also sums all blocks for K)
  const int upto = (b == 0) ? nblk : b;
  int c = 0;
  for (int t = tid; t < upto; t += kUnionThreads) c += counts[t];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) c += __shfl_xor(c, o, 64);
  if (lane == 0) part[wave] = c;
  if (wave == 0) {  // the block's words and their exclusive prefix of member counts
    const uint32_t w = bits[static_cast<int64_t>(b) * kBlkWords + lane];
    word[lane] = w;
    int x = __popc(w);
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {  // inclusive scan across the wavefront
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    wrank[lane] = x - __popc(w);
  }
  __syncthreads();
  int before = 0;
#pragma unroll
  for (int k = 0; k < kUnionThreads / 64; ++k) before += part[k];
  if (b == 0 && tid == 0) {
    u_ids[0] = blank;
    *K_out = 1 + before;  // block 0 summed every block
  }
  const int base = (b == 0) ? 1 : 1 + before;  // first rank of this block's members
  for (int v = lo + tid; v < hi; v += kUnionThreads) {
    const int r = v - lo;
    const uint32_t w = word[r >> 5];
    const uint32_t m = 1u << (r & 31);
    int out = -1;
    if (v == blank) {
      out = 0;
    } else if (w & m) {
      out = base + wrank[r >> 5] + __popc(w & (m - 1u));
      u_ids[out] = v;
    }
    remap[v] = out;
  }
  for (int i = tid; i < total; i += kUnionThreads) {
    const int v = targets[i];
    if (v >= lo && v < hi && v != blank) {
      const int r = v - lo;
      const uint32_t w = word[r >> 5];
      y_rel[i] = base + wrank[r >> 5] + __popc(w & ((1u << (r & 31)) - 1u));
    } else if (b == 0 && (v < 0 || v >= V || v == blank)) {
      y_rel[i] = -1;  // not a label: no block owns it
    }
  }
}

static int union_blocks(int32_t V) { return (V + kBlk - 1) / kBlk; }

size_t union_scratch_bytes(int32_t V) {
  const size_t nblk = static_cast<size_t>(union_blocks(V > 0 ? V : 1));
  return align_up(nblk * kBlkWords * sizeof(uint32_t), 256) + align_up(nblk * sizeof(int32_t), 256);
}

hipError_t launch_union_remap(const int32_t* targets, int32_t total, int32_t blank, int32_t V, int32_t* remap,
                              int32_t* u_ids, int32_t* y_rel, int32_t* K, int32_t* err, void* scratch,
                              hipStream_t stream) {
  const int nblk = union_blocks(V);
  uint32_t* bits = static_cast<uint32_t*>(scratch);
  int32_t* counts = reinterpret_cast<int32_t*>(static_cast<char*>(scratch) +
                                               align_up(static_cast<size_t>(nblk) * kBlkWords * sizeof(uint32_t), 256));
  Prof p("union_remap", stream);
  hipLaunchKernelGGL(union_mark_kernel, dim3(nblk), dim3(kUnionThreads), 0, stream, targets, total, blank, V, bits,
                     counts, err);
  hipLaunchKernelGGL(union_rank_kernel, dim3(nblk), dim3(kUnionThreads), 0, stream, targets, total, blank, V, bits,
                     counts, nblk, remap, u_ids, y_rel, K);
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
