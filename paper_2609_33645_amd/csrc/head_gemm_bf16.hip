// bf16 vocabulary-head products of Pruned CTC on the direct-to-LDS matrix-core engine
// (gemm_bf16.h).  Same computations as the generic kernels in head_gemm.hip:
//  * lse_partial: Z^T tile = W H^T with the online log-sum-exp epilogue (Eq. lognorm;
//    Algorithm 1 online log-sum-exp over vocabulary chunks);
//  * gather_s:    S = Z[:, U] - lambda, subtraction in double, one rounding to float
//    (Algorithm 1; App. B.1 "Forward computation");
//  * recompute_dz: dZ = scatter_U(G) - g p for one vocabulary chunk (Eq. vjp);
//  * dh_gemm: dH partial += dZ W_c;  dw_gemm: dW_c = dZ^T H  (App. A, Step 3).
// Layouts in LDS follow global memory: W and H rows and dZ rows are K-contiguous for the
// forward/recompute/dH-left operands; W (for dH) and dZ, H (for dW) are consumed
// transposed through the LDS transpose read.
#include <type_traits>

#include "gemm_bf16.h"
#include "pctc_internal.h"

namespace pctc {

using bf::GOp;
using bf::LL;

namespace {

constexpr int kFR = 256;  // vocabulary rows per forward/recompute tile
constexpr int kFC = 128;  // frames per forward/recompute tile
constexpr int kFK = 32;   // k per stage
constexpr int kBR = 256;  // backward tile rows (dH: frames, dW: vocabulary)
constexpr int kBC = 256;  // backward tile columns (D)
constexpr int kBK = 32;

// 4 wavefronts (2 x 2), two workgroups per CU so that one's epilogue overlaps the
// other's products
using GFwd = bf::Gemm<kFR, kFC, kFK, LL::KC, LL::KC, 3>;
// the same tiles over gathered W rows (selected classes): flat per-lane addresses
using GFwdGather = bf::Gemm<kFR, kFC, kFK, LL::KC, LL::KC, 3, 2, 2, false, false>;
// 8 wavefronts (2 x 4) on the ping-pong schedule; dZ copied 64 deep (whole 128-byte lines per
// frame row), W 32 deep
using GDh = bf::GemmA64<2, 4>;
// logit products of wide heads (D >= kWideD: normaliser, argmax, recompute): the k loop is
// long enough that the epilogue is a small share, so one 8-wave 256 x 256 workgroup per CU
// beats two 4-wave ones
using GWide = bf::Gemm<256, 256, 64, LL::KC, LL::KC, 2, 2, 4>;
// normaliser and argmax of narrow heads (D < kWideD): 8-wave 256 x 256 tiles, four 32-deep
// stages, runs of kMidRun vocabulary tiles per workgroup (the copy pipeline runs through a
// run, so one workgroup per CU still keeps the matrix pipe fed across tile boundaries)
using GMid = bf::Gemm<256, 256, 32, LL::KC, LL::KC, 4, 2, 4, true>;
// the same tiles with the frame operand read from the transposed head input Ht [D][Mp] (whole
// 512-byte k-lines per copy instead of 64-byte row pieces, i.e. half cache lines): the
// narrow-head dense recompute; the narrow-head normaliser also copies its W rows 64 deep (whole
// 128-byte lines; 3-4% faster there, but 3-5% slower in the recompute, whose W rows come two
// k-tiles ahead instead of three)
using GMidT = bf::Gemm<256, 256, 32, LL::KC, LL::MC, 4, 2, 4, true>;
using GMidTW = bf::GemmMidA64<2, 4>;
constexpr int kMidRun = 8;
constexpr int kRcCus = 224;  // workgroups of the dense recompute (one round)
constexpr int kRcStores = 16;  // buffer stores per wave per 256 x 256 tile (recompute, E)
// the union-column part's dH product: 4-wave tiles (two workgroups per CU), so that its
// workgroups find room beside a recompute's
using GUh = bf::Gemm<256, 128, 32, LL::KC, LL::MC, 3, 2, 2>;
using GDw = bf::Gemm<kBR, kBC, kBK, LL::MC, LL::MC, 4, 2, 4, true>;

__device__ __forceinline__ int xcd_swz(int bid, int nblocks) {
  const int full = (nblocks / 8) * 8;
  if (bid >= full) return bid;
  return (bid % 8) * (full / 8) + bid / 8;
}

// Tile order for an nA x nB grid of output tiles, A = frame tiles (few), B = vocabulary
// tiles or partitions (many).  Consecutive work ids walk groups of ga x gb tiles (a
// fastest) with about 64 tiles per group (what one XCD runs at a time) and ga ~ 11 frame
// tiles; the groups walk the frame groups fastest, so the few groups that cover every frame
// tile of a run of vocabulary rows are consecutive: that XCD fetches the rows once and the
// frame tiles (the small operand) stay in its L2.  Grid = ceil(nA/ga) ga * ceil(nB/gb) gb;
// ids past the edge return false.
__host__ __device__ __forceinline__ void group_shape(int nA, int& ga, int& gb) {
  const int groups = (nA + 10) / 11;
  ga = (nA + groups - 1) / groups;
  gb = 64 / ga;
  if (gb < 1) gb = 1;
}
__host__ __device__ __forceinline__ int grouped_grid(int nA, int nB) {
  int ga, gb;
  group_shape(nA, ga, gb);
  return ((nA + ga - 1) / ga) * ga * ((nB + gb - 1) / gb) * gb;
}
__device__ __forceinline__ bool grouped_tile(int work, int nA, int nB, int& a, int& b) {
  int ga, gb;
  group_shape(nA, ga, gb);
  const int gA = (nA + ga - 1) / ga;
  const int blk = work / (ga * gb), in = work % (ga * gb);
  a = (blk % gA) * ga + in % ga;
  b = (blk / gA) * gb + in / ga;
  return a < nA && b < nB;
}

// Accumulators of a tile start at the bias of their row (bt: the tile's rows, in LDS).
template <int FR, int FC, class G = GFwd>
__device__ __forceinline__ void bias_init(f32x16 (&acc)[FR][FC], const float* bt, int wave, int lane) {
#pragma unroll
  for (int i = 0; i < FR; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 b4 = *reinterpret_cast<const float4*>(bt + G::row_of(wave, lane, i, 4 * q));
#pragma unroll
      for (int j = 0; j < FC; ++j) {
        acc[i][j][4 * q + 0] = b4.x;
        acc[i][j][4 * q + 1] = b4.y;
        acc[i][j][4 * q + 2] = b4.z;
        acc[i][j][4 * q + 3] = b4.w;
      }
    }
}

// Logits of rows at or past vend (a partition's ragged last tile, whose rows read as zeros)
// become -inf in place, so that the update below treats every tile alike.  Each row test is
// used at once for the FC columns it covers (a lane holds 4 consecutive rows per group):
// keeping one test per accumulator live across both passes of the update would take a mask
// register pair per element.
template <int FR, int FC, class G = GFwd>
__device__ __forceinline__ void mask_rows_inf(f32x16 (&acc)[FR][FC], int v0, int vend, int wave, int lane) {
#pragma unroll
  for (int i = 0; i < FR; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int lim = vend - v0 - G::row_of(wave, lane, i, 4 * q);  // rows e < lim are in range
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool out = e >= lim;
#pragma unroll
        for (int j = 0; j < FC; ++j) acc[i][j][4 * q + e] = out ? -INFINITY : acc[i][j][4 * q + e];
      }
    }
}

// Online log-sum-exp update of the running (max, sum) of this lane's frames with one
// tile of logits (bias included; out-of-range rows already -inf).
template <int FR, int FC, class G = GFwd>
__device__ __forceinline__ void lse_tile_update(const f32x16 (&acc)[FR][FC], float (&run_max)[FC],
                                                float (&run_sum)[FC]) {
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

}  // namespace

#define PCTC_STAGES_G(G)                                                                  \
  __shared__ __attribute__((aligned(1024))) char st0_[G::kKernelStageBytes];                      \
  __shared__ __attribute__((aligned(1024))) char st1_[G::kKernelStageBytes];                      \
  __shared__ __attribute__((aligned(1024))) char st2_[G::kNS >= 3 ? G::kKernelStageBytes : 16];   \
  __shared__ __attribute__((aligned(1024))) char st3_[G::kNS >= 4 ? G::kKernelStageBytes : 16];   \
  char* const stx_[4] = {st0_, st1_, st2_, st3_};                                           \
  char* const(&st)[G::kNS] = *reinterpret_cast<char* const(*)[G::kNS]>(&stx_);

// The two wavefronts of each frame column (row halves) combine their running (max, sum)
// pairs through LDS (xch: any drained stage) and write the partition's pair of every frame.
template <class G>
__device__ __forceinline__ void lse_store_partials(const float (&run_max)[G::FC], const float (&run_sum)[G::FC],
                                                   char* xchb, int wave, int lane, int m0, int M,
                                                   float2* __restrict__ out) {
  constexpr int FC = G::FC;
  __syncthreads();
  constexpr int WC = G::NW / 2;  // column groups (the wave grid is 2 x WC)
  float2* xch = reinterpret_cast<float2*>(xchb);
  const int rowhalf = wave / WC, colq = wave % WC;
  if (rowhalf == 1 && lane < 32) {
#pragma unroll
    for (int j = 0; j < FC; ++j) xch[colq * (FC * 32) + j * 32 + lane] = make_float2(run_max[j], run_sum[j]);
  }
  __syncthreads();
  if (rowhalf == 0 && lane < 32) {
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      const float2 o = xch[colq * (FC * 32) + j * 32 + lane];
      const float nmax = fmaxf(run_max[j], o.x);
      float s = 0.f;
      if (run_max[j] != -INFINITY) s += run_sum[j] * fast_exp2((run_max[j] - nmax) * kLog2e);
      if (o.x != -INFINITY) s += o.y * fast_exp2((o.x - nmax) * kLog2e);
      if (nmax != nmax) s = nmax;
      const int m = m0 + G::col_of(wave, lane, j);
      if (m < M) out[m] = make_float2(nmax, s);
    }
  }
}

template <class G, bool BIAS, int OCC>
__global__ void __launch_bounds__(G::kThreads, OCC)
lse_partial_bf16(const uint16_t* __restrict__ H, int M, int D, const uint16_t* __restrict__ W, const float* __restrict__ bias,
                 int V, int P, int vper, float2* __restrict__ partials) {
  extern __shared__ float bsh[];  // BIAS: b over this partition's rows (vper, padded to whole tiles)
  constexpr int FR = G::FR, FC = G::FC, TR = G::kBR, TC = G::kBC;
  PCTC_STAGES_G(G)
  const int nMt = (M + TC - 1) / TC;
  // every frame tile of a vocabulary run on one XCD at about the same time: the run's W rows
  // are fetched once and shared through that XCD's L2
  const int w = xcd_swz(blockIdx.x, gridDim.x);
  const int mt = w % nMt;
  const int p = w / nMt;
  if (p >= P) return;
  const int m0 = mt * TC;
  const int vbeg = p * vper;
  const int vend = min(V, vbeg + vper);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ntiles = (vend - vbeg + TR - 1) / TR;
  if (BIAS) {
    // visible to every wave after the engine's first barrier
    for (int r = tid; r < ntiles * TR; r += G::kThreads) bsh[r] = (vbeg + r < vend) ? bias[vbeg + r] : 0.f;
    __syncthreads();
  }
  const GOp A{W, D, vend, D, nullptr};
  const GOp B{H, D, M, D, nullptr};
  float run_max[FC], run_sum[FC];
#pragma unroll
  for (int j = 0; j < FC; ++j) {
    run_max[j] = -INFINITY;
    run_sum[j] = 0.f;
  }
  f32x16 acc[FR][FC];
  auto epi = [&](int i, f32x16 (&a)[FR][FC]) {
    const int v0 = vbeg + i * TR;
    if (v0 + TR > vend) mask_rows_inf<FR, FC, G>(a, v0, vend, wave, lane);
    lse_tile_update<FR, FC, G>(a, run_max, run_sum);
  };
  if (BIAS)
    G::run_seq(A, B, vbeg, m0, ntiles, D, st, acc, epi, [&](int i, f32x16 (&a)[FR][FC]) {
      bias_init<FR, FC, G>(a, bsh + i * TR, wave, lane);
    });
  else
    G::run_seq(A, B, vbeg, m0, ntiles, D, st, acc, epi);
  lse_store_partials<G>(run_max, run_sum, st0_, wave, lane, m0, M, partials + static_cast<int64_t>(p) * M);
}

// Log-sum-exp update of one frame column of an E tile (lse_partial_e_bf16) with the pair
// (0, s): s is this lane's sum of exp(z) over its rows, the other lane half's rows are added
// here; when the tile's sum leaves [2^-100, 2^100] the maximum-based update is taken on the
// same logits instead (the decision is the same on both lane halves).
template <int FR, int FC>
__device__ __forceinline__ void lse_e_update(const f32x16 (&a)[FR][FC], int j, float s, float& run_max,
                                             float& run_sum) {
  float sj = s + swap_halves(s);
  float mj = 0.f;
  if (!(sj >= 0x1p-100f && sj <= 0x1p100f)) {
    float tmax = -INFINITY;
#pragma unroll
    for (int i = 0; i < FR; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, a[i][j][r]);
    tmax = fmaxf(tmax, swap_halves(tmax));
    const float ms = (tmax == -INFINITY) ? 0.f : tmax * kLog2e;
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < FR; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) t += fast_exp2(fmaf(a[i][j][r], kLog2e, -ms));
    sj = t + swap_halves(t);
    mj = tmax;
  }
  const float nmax = fmaxf(run_max, mj);
  float acc_s = 0.f;
  if (run_max != -INFINITY) acc_s += run_sum * fast_exp2((run_max - nmax) * kLog2e);
  if (mj != -INFINITY) acc_s += sj * fast_exp2((mj - nmax) * kLog2e);
  run_sum = acc_s;
  run_max = nmax;
}

// The normaliser of a narrow head (8-wave 256 x 256 tiles, no bias) that also writes, for the
// vocabulary rows of the first eparts partitions (the backward's first chunk), E = exp(z) in
// bf16 into the gradient buffer, laid out like dZ (E[m * epitch + v]); the backward then needs
// no recompute for that chunk: its dense part -g_m p_v(m) = s_m E[m][v] with the per-frame
// scale s_m = -g_m exp(-lambda_m) (hs_scale_bf16).  On those partitions the log-sum-exp is
// taken on the same exponentials with 0 as the reference instead of the running maximum
// (the pair (0, sum exp z) is exact as long as the sum stays in range; a column whose tile
// sum leaves [2^-100, 2^100] takes the maximum-based update instead).  E itself is usable
// when every lambda_m lies in [kEMin, kEMax] (no bf16 overflow, no significant underflow); the
// finalize checks that and the backward recomputes the chunk otherwise.  E partitions run the
// aligned tile sequence (the stores drain under the next tile's products); the others run
// exactly like lse_partial_bf16.  einv (the check flag) is cleared here, before the finalize
// sets it.
// HT: the frames come from Ht [D][Mp] (the transposed head input) instead of H [M][D].
template <bool HT>
__global__ void __launch_bounds__(512, 1)
lse_partial_e_bf16(const uint16_t* __restrict__ H, const uint16_t* __restrict__ Ht, int Mp, int M, int D,
                   const uint16_t* __restrict__ W, int V, int P, int vper, float2* __restrict__ partials,
                   uint16_t* __restrict__ E, int epitch, int eparts, int32_t* __restrict__ einv) {
  using G = std::conditional_t<HT, GMidTW, GMid>;
  constexpr int FR = G::FR, FC = G::FC, TR = G::kBR, TC = G::kBC;
  static_assert(FR == 4 && FC == 2 && G::NW == 8 && TR == 256, "waves of 128 vocabulary rows x 64 frames");
  PCTC_STAGES_G(G)
  __shared__ __attribute__((aligned(1024))) char stg_[G::NW * 4096];
  const int nMt = (M + TC - 1) / TC;
  const int w = xcd_swz(blockIdx.x, gridDim.x);
  const int mt = w % nMt;
  const int p = w / nMt;
  if (blockIdx.x == 0 && threadIdx.x == 0) *einv = 0;
  if (p >= P) return;
  const int m0 = mt * TC;
  const int vbeg = p * vper;
  const int vend = min(V, vbeg + vper);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int ntiles = (vend - vbeg + TR - 1) / TR;
  const GOp A{W, D, vend, D, nullptr};
  const GOp B = HT ? GOp{Ht, Mp, M, D, nullptr} : GOp{H, D, M, D, nullptr};
  float run_max[FC], run_sum[FC];
#pragma unroll
  for (int j = 0; j < FC; ++j) {
    run_max[j] = -INFINITY;
    run_sum[j] = 0.f;
  }
  f32x16 acc[FR][FC];
  if (p >= eparts) {
    auto epi = [&](int i, f32x16 (&a)[FR][FC]) {
      const int v0 = vbeg + i * TR;
      if (v0 + TR > vend) mask_rows_inf<FR, FC, G>(a, v0, vend, wave, lane);
      lse_tile_update<FR, FC, G>(a, run_max, run_sum);
    };
    if constexpr (HT) G::template seq_aligned<0>(A, B, vbeg, m0, ntiles, D, acc, epi);
    else G::run_seq(A, B, vbeg, m0, ntiles, D, st, acc, epi);
  } else {
    const int wr = wave / (G::NW / 2), wc = wave % (G::NW / 2);
    const uint64_t zb = reinterpret_cast<uint64_t>(E + static_cast<int64_t>(m0) * epitch);
    const uint64_t zbu =
        (static_cast<uint64_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(zb >> 32))) << 32) |
        static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(zb)));
    const int zsize = __builtin_amdgcn_readfirstlane(min(M - m0, TC) * epitch * 2);
    const __amdgpu_buffer_rsrc_t zr = __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(zbu),
                                                                       static_cast<short>(0), zsize, bf::kBufWord3);
    char* const stg = stg_ + wave * 4096;
    const int rf = lane & 31, hl = lane >> 5;
    auto epi = [&](int it, f32x16 (&a)[FR][FC]) {
      const int v0 = vbeg + it * TR;
      if (v0 + TR > vend) mask_rows_inf<FR, FC, G>(a, v0, vend, wave, lane);
      const int vb = v0 + (TR / 2) * wr;  // this wave's first vocabulary row
      float s[FC] = {0.f, 0.f};
#pragma unroll
      for (int h = 0; h < 4; ++h) {  // frames 32 j.. of the wave, vocabulary blocks ib, ib + 1
        const int j = h >> 1, ib = 2 * (h & 1);
#pragma unroll
        for (int il = 0; il < 2; ++il)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = fast_exp2(a[ib + il][j][4 * q + e] * kLog2e);
            s[j] += (v[0] + v[1]) + (v[2] + v[3]);
            const int c = 32 * il + 8 * q + 4 * hl;
            const int off = rf * 128 + (((c >> 3) ^ (rf & 7)) << 4) + (((c >> 2) & 1) << 3);
            *reinterpret_cast<u32x2*>(stg + off) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
          }
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int f = (lane >> 3) + 8 * t, slot = lane & 7;
          const u32x4 val = *reinterpret_cast<const u32x4*>(stg + f * 128 + ((slot ^ (f & 7)) << 4));
          const int row = 64 * wc + 32 * j + f;
          const uint32_t off = static_cast<uint32_t>(row * epitch + vb + 64 * (h & 1) + 8 * slot) * 2u;
          __builtin_amdgcn_raw_buffer_store_b128(val, zr, off, 0, 2 /* nt: read back only by dH and dW */);
        }
        if (h & 1) lse_e_update(a, j, s[j], run_max[j], run_sum[j]);  // column j's logits are done with
      }
    };
    if constexpr (HT) G::template seq_aligned<kRcStores>(A, B, vbeg, m0, ntiles, D, acc, epi);
    else G::template run_seq_aligned<kRcStores>(A, B, vbeg, m0, ntiles, D, st, acc, epi);
  }
  lse_store_partials<G>(run_max, run_sum, stg_, wave, lane, m0, M, partials + static_cast<int64_t>(p) * M);
}

// ---------------------------------------------------------------------------------------
// Greedy emission head: framewise argmax of H W^T (+ b) over a vocabulary partition, on the
// same pipelined tiles as the normaliser.  Within a lane the rows are visited in
// increasing order and only a strictly larger logit replaces the best, so ties keep the
// smallest class id; the combines below keep that rule.
// ---------------------------------------------------------------------------------------
__device__ __forceinline__ void amax_merge(float& bv, int& bi, float ov, int oi) {
  if (ov > bv || (ov == bv && oi < bi)) {
    bv = ov;
    bi = oi;
  }
}

template <class G, bool BIAS, int OCC>
__global__ void __launch_bounds__(G::kThreads, OCC)
amax_partial_bf16(const uint16_t* __restrict__ H, int M, int D, const uint16_t* __restrict__ W,
                  const float* __restrict__ bias, int V, int P, int vper, float2* __restrict__ partials) {
  extern __shared__ float bsh[];  // BIAS: b over this partition's rows
  constexpr int FR = G::FR, FC = G::FC, TR = G::kBR, TC = G::kBC;
  PCTC_STAGES_G(G)
  const int nMt = (M + TC - 1) / TC;
  int mt, p;
  if (!grouped_tile(xcd_swz(blockIdx.x, gridDim.x), nMt, P, mt, p)) return;
  const int m0 = mt * TC;
  const int vbeg = p * vper;
  const int vend = min(V, vbeg + vper);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ntiles = (vend - vbeg + TR - 1) / TR;
  if (BIAS) {
    for (int r = tid; r < ntiles * TR; r += G::kThreads) bsh[r] = (vbeg + r < vend) ? bias[vbeg + r] : 0.f;
    __syncthreads();
  }
  const GOp A{W, D, vend, D, nullptr};
  const GOp B{H, D, M, D, nullptr};
  float bv[FC];
  int bi[FC];
#pragma unroll
  for (int j = 0; j < FC; ++j) {
    bv[j] = -INFINITY;
    bi[j] = 0x7fffffff;
  }
  f32x16 acc[FR][FC];
  auto epi = [&](int it, f32x16 (&a)[FR][FC]) {
    const int v0 = vbeg + it * TR;
    if (v0 + TR > vend) mask_rows_inf<FR, FC, G>(a, v0, vend, wave, lane);  // -inf never replaces the best
    // the lane's rows increase with (i, r): the tile's best is its largest logit at the first
    // row holding it (found scanning backwards), and it replaces the running best only when
    // strictly larger, so ties keep the smallest id; NaN never compares equal or larger
    const int rbase = v0 + G::row_of(wave, lane, 0, 0);
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      float tmax = -INFINITY;
#pragma unroll
      for (int i = 0; i < FR; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, a[i][j][r]);
      int off = 0;
#pragma unroll
      for (int i = FR - 1; i >= 0; --i)
#pragma unroll
        for (int r = 15; r >= 0; --r) off = (a[i][j][r] == tmax) ? 32 * i + 8 * (r >> 2) + (r & 3) : off;
      if (tmax > bv[j]) {
        bv[j] = tmax;
        bi[j] = rbase + off;
      }
    }
  };
  if (BIAS)
    G::run_seq(A, B, vbeg, m0, ntiles, D, st, acc, epi, [&](int it, f32x16 (&a)[FR][FC]) {
      bias_init<FR, FC, G>(a, bsh + it * TR, wave, lane);
    });
  else
    G::run_seq(A, B, vbeg, m0, ntiles, D, st, acc, epi);
  // lane halves hold the other half of each 32-row block, then the row halves of the tile
#pragma unroll
  for (int j = 0; j < FC; ++j) {
    const float ov = swap_halves(bv[j]);
    const int oi = __shfl_xor(bi[j], 32, 64);
    amax_merge(bv[j], bi[j], ov, oi);
  }
  __syncthreads();
  float2* xch = reinterpret_cast<float2*>(st0_);
  constexpr int WC = G::NW / 2;  // column groups (the wave grid is 2 x WC)
  const int rowhalf = wave / WC, colq = wave % WC;
  if (rowhalf == 1 && lane < 32) {
#pragma unroll
    for (int j = 0; j < FC; ++j)
      xch[colq * (FC * 32) + j * 32 + lane] = make_float2(bv[j], __int_as_float(bi[j]));
  }
  __syncthreads();
  if (rowhalf == 0 && lane < 32) {
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      const float2 o = xch[colq * (FC * 32) + j * 32 + lane];
      amax_merge(bv[j], bi[j], o.x, __float_as_int(o.y));
      const int m = m0 + G::col_of(wave, lane, j);
      if (m < M) partials[static_cast<int64_t>(p) * M + m] = make_float2(bv[j], __int_as_float(bi[j]));
    }
  }
}

__global__ void __launch_bounds__(256, 2)
gather_s_bf16(const uint16_t* __restrict__ H, int M, int D, const uint16_t* __restrict__ W,
              const float* __restrict__ bias, const int32_t* __restrict__ u_ids, const int32_t* __restrict__ Kdev,
              const double* __restrict__ lam, float* __restrict__ S, int ldS, double* __restrict__ Zd) {
  using G = GFwdGather;
  constexpr int FR = G::FR, FC = G::FC;
  PCTC_STAGES_G(G)
  const int nMt = (M + kFC - 1) / kFC;
  const int mt = blockIdx.x % nMt;
  const int jt = blockIdx.x / nMt;
  const int K = *Kdev;
  const int j0 = jt * kFR;
  if (j0 >= K) return;
  const int m0 = mt * kFC;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const GOp A{W, D, K, D, u_ids};
  const GOp B{H, D, M, D, nullptr};
  f32x16 acc[FR][FC];
  G::run(A, B, j0, m0, 0, D, st, acc);
#pragma unroll
  for (int j = 0; j < FC; ++j) {
    const int m = m0 + GFwd::col_of(wave, lane, j);
    if (m >= M) continue;
    const double l = Zd ? 0.0 : lam[m];
#pragma unroll
    for (int i = 0; i < FR; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int jj = j0 + GFwd::row_of(wave, lane, i, r);
        if (jj < K) {
          double z = static_cast<double>(acc[i][j][r]);
          if (bias) z += static_cast<double>(bias[u_ids[jj]]);
          if (Zd)  // the logit itself; lambda is subtracted once it is known
            Zd[static_cast<int64_t>(m) * ldS + jj] = z;
          else
            S[static_cast<int64_t>(m) * ldS + jj] = static_cast<float>(z - l);
        }
      }
  }
}

// dZ chunk [M][chunk] (row pitch `chunk`): dZ[m][v] = scatter_U(G)[m][v] - g_m p_v(m) for
// the chunk's 256-column tiles (Eq. vjp; zero on excluded frames).  The dense part -g p
// comes from the recomputed logits of Hs (H with excluded rows zeroed, so their products
// are finite and, with g_m = 0, give zeros) plus the bias when there is one; the few union
// columns of a tile are then rewritten in the staging buffer as G[m][j] - g_m exp(S[m][j])
// from the forward's selected log-probabilities.  Columns past cw within the last tile
// hold finite values that no consumer reads (their W rows read as zero).  Each tile (256
// vocabulary rows x 128 or 256 frames) is staged through the drained LDS stages, 32 frames
// of each 64-frame column group per pass, so that every frame row is stored as contiguous
// 16-byte vectors.  DB: the staged (rounded) values are also summed
// over the tile's frames, giving this tile's share of db = dZ^T 1 in
// dbpart[frame tile][column].
template <class GG, bool BIAS, bool DB, int OCC>
__global__ void __launch_bounds__(GG::kThreads, OCC)
recompute_dz_bf16(const uint16_t* __restrict__ Hs, int M, int D, const uint16_t* __restrict__ W,
                  const float* __restrict__ bias, int c0, int cw, const float2* __restrict__ lam2,
                  const float* __restrict__ g, const int32_t* __restrict__ remap, const float* __restrict__ S, int ldS,
                  const float* __restrict__ G, int ldG, uint16_t* __restrict__ dZ, int chunk,
                  float* __restrict__ dbpart) {
  constexpr int FR = GG::FR, FC = GG::FC, TR = GG::kBR, TC = GG::kBC, NT = GG::kThreads;
  static_assert(TR == 256 && NT % TR == 0, "each thread owns one tile column");
  constexpr int WC = GG::NW / 2;        // column groups of 64 frames (the wave grid is 2 x WC)
  constexpr int kPitch = TR * 2 + 16;  // staging row: 256 bf16 + 16 bytes
  // in each pass, column group q stages its 32 frames in stage q / kGps, row block q % kGps
  // (the k loop has drained, so every stage is free)
  constexpr int kGps = GG::kStageBytes / (32 * kPitch);
  static_assert(kGps >= 1 && (WC + kGps - 1) / kGps <= GG::kNS, "staging fits the stages");
  PCTC_STAGES_G(GG)
  const int nMt = (M + TC - 1) / TC;
  const int nVt = (cw + TR - 1) / TR;
  int mt, vt;
  if (!grouped_tile(xcd_swz(blockIdx.x, gridDim.x), nMt, nVt, mt, vt)) return;
  const int m0 = mt * TC;
  const int vl0 = vt * TR;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // union columns of this tile: (union index << 8) | tile column; b per column
  __shared__ int ulist[TR];
  __shared__ int nu;
  __shared__ __attribute__((aligned(16))) float bl[BIAS ? TR : 4];
  __shared__ float dbx[(DB && NT > TR) ? NT - TR : 1];
  if (tid == 0) nu = 0;
  const bool vin = tid < TR && vl0 + tid < cw;
  const int jsel = (vin && remap) ? remap[c0 + vl0 + tid] : -1;  // no remap: dense part only
  if (BIAS && tid < TR) bl[tid] = vin ? bias[c0 + vl0 + tid] : 0.f;
  const int any_sel = __syncthreads_or(jsel >= 0);
  if (any_sel) {
    if (jsel >= 0) ulist[atomicAdd(&nu, 1)] = (jsel << 8) | tid;
    __syncthreads();
  }
  // this lane's frames: -g_m p = -sign(g_m) 2^(z log2(e) - (lambda_m log2(e) - log2|g_m|)), so
  // the exponent offset ll takes g_m's magnitude (+inf on excluded frames, whose products
  // are finite: the values are zeros) and sg its sign, applied to a packed bf16 pair
  float ll[FC];
  uint32_t sg[FC];
#pragma unroll
  for (int j = 0; j < FC; ++j) {
    const int m = m0 + GG::col_of(wave, lane, j);
    const float gm = (m < M) ? g[m] : 0.f;
    const float2 l2 = (m < M) ? lam2[m] : make_float2(0.f, 0.f);
    ll[j] = (gm != 0.f) ? (l2.x + l2.y) - fast_log2(fabsf(gm)) : INFINITY;
    sg[j] = (gm > 0.f) ? 0x80008000u : 0u;
  }
  const GOp A{W + static_cast<int64_t>(c0) * D, D, cw, D, nullptr};
  const GOp B{Hs, D, M, D, nullptr};
  f32x16 acc[FR][FC];
  if (BIAS) {  // the logits' accumulators start at b (visible after the barrier above)
    bias_init<FR, FC, GG>(acc, bl, wave, lane);
    GG::template run<false>(A, B, vl0, m0, 0, D, st, acc);
  } else {
    GG::run(A, B, vl0, m0, 0, D, st, acc);
  }
  auto stage_of = [&](int q) -> char* {
    const int sq = q / kGps;
    char* const b = (sq == 0) ? st0_ : (sq == 1) ? st1_ : (sq == 2) ? st2_ : st3_;
    return b + (q % kGps) * (32 * kPitch);
  };
  const int nunion = any_sel ? nu : 0;
  char* stage = stage_of(wave % WC);  // this wave's frames [64 q, 64 q + 64) of the tile, 32 per pass
  // DB: column tid % 256 of the tile over column groups [qb, qb + kQPer), summed over the passes
  constexpr int kQPer = WC / (NT / TR);
  const int qb = (tid / TR) * kQPer;
  float dbsum = 0.f;
#pragma unroll
  for (int j = 0; j < FC; ++j) {
    if (j > 0) __syncthreads();  // the previous pass's readers are done
#pragma unroll
    for (int i = 0; i < FR; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int rl0 = GG::row_of(wave, lane, i, 4 * q);
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = fast_exp2(fmaf(acc[i][j][4 * q + e], kLog2e, -ll[j]));
        *reinterpret_cast<u32x2*>(stage + (lane & 31) * kPitch + rl0 * 2) =
            u32x2{pack_bf16x2(v[0], v[1]) ^ sg[j], pack_bf16x2(v[2], v[3]) ^ sg[j]};
      }
    __syncthreads();
    if (nunion > 0) {
      // the union columns of the WC x 32 staged frames
      for (int idx = tid; idx < nunion * (WC * 32); idx += NT) {
        const int e = ulist[idx / (WC * 32)];
        const int col = e & 255, ju = e >> 8;
        const int grp = (idx >> 5) % WC, row = idx & 31;
        const int m = m0 + 64 * grp + 32 * j + row;
        float val = 0.f;
        if (m < M) {
          const float gm = g[m];
          if (gm != 0.f)
            val = G[static_cast<int64_t>(m) * ldG + ju] - gm * fast_exp2(S[static_cast<int64_t>(m) * ldS + ju] * kLog2e);
        }
        *reinterpret_cast<uint16_t*>(stage_of(grp) + row * kPitch + col * 2) = f32_to_bf16(val);
      }
      __syncthreads();
    }
    if (DB) {
      // column tid % 256 over this thread's staged frames (frames past M hold zeros)
      const int col = tid % TR;
#pragma unroll 4
      for (int row = 0; row < 32; ++row)
#pragma unroll
        for (int q = 0; q < kQPer; ++q)
          dbsum += bf16_to_f32(*reinterpret_cast<const uint16_t*>(stage_of(qb + q) + row * kPitch + col * 2));
    }
    // WC groups x 32 frames x 32 vectors of 16 bytes
#pragma unroll
    for (int k = 0; k < (WC * 1024) / NT; ++k) {
      const int idx = tid + NT * k;
      const int grp = idx >> 10;
      const int row = (idx >> 5) & 31;
      const int vec = idx & 31;
      const int mm = m0 + 64 * grp + 32 * j + row;
      const char* src = stage_of(grp) + row * kPitch + vec * 16;
      const u32x4 v = *reinterpret_cast<const u32x4*>(src);
      // streaming store: dZ is read back only by the next two products, and keeping its
      // lines out of the caches leaves them to those products' operands
      if (mm < M)
        __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(dZ + static_cast<int64_t>(mm) * chunk + vl0 + vec * 8));
    }
  }
  if (DB) {
    if constexpr (NT > TR) {  // the other threads of each column hand over their share
      if (tid >= TR) dbx[tid - TR] = dbsum;
      __syncthreads();
      if (tid < TR) {
#pragma unroll
        for (int p = 1; p < NT / TR; ++p) dbsum += dbx[(p - 1) * TR + tid];
      }
    }
    if (tid < TR) dbpart[static_cast<int64_t>(mt) * chunk + vl0 + tid] = dbsum;
  }
}

// The dense part -g p of one chunk (no bias, no db, no union columns) on the normaliser's
// 8-wave 256 x 256 tiles, `run` vocabulary tiles per workgroup: the copy pipeline runs
// through the run, so the next tile's copies land while this tile's epilogue runs.  The
// epilogue needs no barrier: each wave stages its own 64-vocabulary x 32-frame blocks (four
// per tile) through a private 4 KB LDS buffer (16-byte slots XOR-swizzled by frame) and
// writes 128 contiguous bytes per frame row with buffer stores.  The stores always issue
// (frames past M fall outside the resource, which drops them), so the copy pipeline can
// count them and leave them in flight under the next tile's first products.

// HT: the frames come from Hst [D][Mp] (Hs transposed) instead of Hs [M][D].
template <bool HT>
__global__ void __launch_bounds__(512, 1)
recompute_run_bf16(const uint16_t* __restrict__ Hs, const uint16_t* __restrict__ Hst, int Mp, int M, int D,
                   const uint16_t* __restrict__ W, int c0, int cw, int run, const float2* __restrict__ lam2,
                   const float* __restrict__ g, uint16_t* __restrict__ dZ, int chunk,
                   const int32_t* __restrict__ only_if) {
  // only_if (the normaliser's E check flag): recompute only when its E cannot be used
  if (only_if && *only_if == 0) return;
  using G = std::conditional_t<HT, GMidT, GMid>;
  constexpr int FR = G::FR, FC = G::FC, TR = G::kBR, TC = G::kBC;
  static_assert(FR == 4 && FC == 2 && G::NW == 8 && TR == 256, "waves of 128 vocabulary rows x 64 frames");
  PCTC_STAGES_G(G)
  __shared__ __attribute__((aligned(1024))) char stg_[G::NW * 4096];
  const int nMt = (M + TC - 1) / TC;
  const int nVt = (cw + TR - 1) / TR;
  // all frame tiles of a vocabulary run consecutive on one XCD (it fetches the run's W rows once)
  const int w = xcd_swz(blockIdx.x, gridDim.x);
  const int mt = w % nMt;
  const int vt0 = (w / nMt) * run;
  if (vt0 >= nVt) return;
  const int ntiles = min(run, nVt - vt0);
  const int m0 = mt * TC;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave / (G::NW / 2), wc = wave % (G::NW / 2);
  // -g_m p = -sign(g_m) 2^(z log2(e) - (lambda_m log2(e) - log2|g_m|)), as in recompute_dz_bf16
  float ll[FC];
  uint32_t sg[FC];
#pragma unroll
  for (int j = 0; j < FC; ++j) {
    const int m = m0 + G::col_of(wave, lane, j);
    const float gm = (m < M) ? g[m] : 0.f;
    const float2 l2 = (m < M) ? lam2[m] : make_float2(0.f, 0.f);
    ll[j] = (gm != 0.f) ? (l2.x + l2.y) - fast_log2(fabsf(gm)) : INFINITY;
    sg[j] = (gm > 0.f) ? 0x80008000u : 0u;
  }
  const GOp A{W + static_cast<int64_t>(c0) * D, D, cw, D, nullptr};
  const GOp B = HT ? GOp{Hst, Mp, M, D, nullptr} : GOp{Hs, D, M, D, nullptr};
  // store resource: this frame tile's rows of dZ (byte offsets < 256 rows x 2 chunk)
  const uint64_t zb = reinterpret_cast<uint64_t>(dZ + static_cast<int64_t>(m0) * chunk);
  const uint64_t zbu = (static_cast<uint64_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(zb >> 32))) << 32) |
                       static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(zb)));
  const int zsize = __builtin_amdgcn_readfirstlane(min(M - m0, TC) * chunk * 2);
  const __amdgpu_buffer_rsrc_t zr =
      __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(zbu), static_cast<short>(0), zsize, bf::kBufWord3);
  char* const stg = stg_ + wave * 4096;
  const int rf = lane & 31, hl = lane >> 5;
  f32x16 acc[FR][FC];
  auto epi = [&](int it, f32x16 (&a)[FR][FC]) {
    const int vb = (vt0 + it) * TR + (TR / 2) * wr;  // this wave's first vocabulary column in the chunk
#pragma unroll
    for (int h = 0; h < 4; ++h) {  // frames 32 j.. of the wave, vocabulary blocks ib, ib + 1
      const int j = h >> 1, ib = 2 * (h & 1);
#pragma unroll
      for (int il = 0; il < 2; ++il)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = fast_exp2(fmaf(a[ib + il][j][4 * q + e], kLog2e, -ll[j]));
          const int c = 32 * il + 8 * q + 4 * hl;  // 4 consecutive vocabulary columns of frame rf
          const int off = rf * 128 + (((c >> 3) ^ (rf & 7)) << 4) + (((c >> 2) & 1) << 3);
          *reinterpret_cast<u32x2*>(stg + off) = u32x2{pack_bf16x2(v[0], v[1]) ^ sg[j], pack_bf16x2(v[2], v[3]) ^ sg[j]};
        }
#pragma unroll
      for (int t = 0; t < 4; ++t) {  // lanes 8 f.. 8 f + 7 take frame row f + 8 t
        const int f = (lane >> 3) + 8 * t, slot = lane & 7;
        const u32x4 val = *reinterpret_cast<const u32x4*>(stg + f * 128 + ((slot ^ (f & 7)) << 4));
        const int row = 64 * wc + 32 * j + f;  // frame within the tile
        const uint32_t off = static_cast<uint32_t>(row * chunk + vb + 64 * (h & 1) + 8 * slot) * 2u;
        __builtin_amdgcn_raw_buffer_store_b128(val, zr, off, 0, 2 /* nt: read back only by dH and dW */);
      }
    }
  };
  G::template run_seq_aligned<kRcStores>(A, B, vt0 * TR, m0, ntiles, D, st, acc, epi);
}

// db[c0 + v] = sum over frame tiles of dbpart[t][v], v < cw (fixed order).
__global__ void db_reduce_bf16(const float* __restrict__ dbpart, int ntiles, int chunk, int cw,
                               float* __restrict__ db) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= cw) return;
  float s = 0.f;
  for (int t = 0; t < ntiles; ++t) s += dbpart[static_cast<int64_t>(t) * chunk + v];
  db[v] = s;
}

// Tile r of an nA x nB grid walked block by block: the grid is cut into ga x (8 / ga) blocks
// (edge blocks smaller), blocks in row order, tiles within a block b fastest.
__device__ __forceinline__ void block_tile(int r, int nA, int nB, int ga, int& a, int& b) {
  const int gb = 8 / ga;
  const int ba = (nA + ga - 1) / ga, bb = (nB + gb - 1) / gb;
  for (int i = 0; i < ga; ++i) {
    const int a0 = i * ba, ha = min(ba, nA - a0);
    if (ha <= 0) break;
    for (int j = 0; j < gb; ++j) {
      const int b0 = j * bb, hb = min(bb, nB - b0);
      if (hb <= 0) break;
      if (r < ha * hb) {
        a = a0 + r / hb;
        b = b0 + r % hb;
        return;
      }
      r -= ha * hb;
    }
  }
  a = nA;  // not reached for r < nA nB
  b = 0;
}

// gm for the dH product: the frame x d partition over 8 XCDs that reads the least (W columns
// are read gm times, dZ rows 8 / gm times).
static int dh_xcd_rows(int M, int D) {
  int best = 8;
  long long cost = -1;
  for (int gm = 1; gm <= 8; gm *= 2) {
    const long long c = static_cast<long long>(gm) * D + static_cast<long long>(8 / gm) * M;
    if (cost < 0 || c < cost) {
      cost = c;
      best = gm;
    }
  }
  return best;
}

template <class G, int OCC>
__global__ void __launch_bounds__(G::kThreads, OCC)
dh_gemm_bf16(const uint16_t* __restrict__ dZ, int M, int chunk, const uint16_t* __restrict__ W, int D, int c0, int cw,
             int slice, float* __restrict__ part, int gm, int accumulate, const int32_t* __restrict__ kdev,
             const float* __restrict__ rowscale) {
  // the first chunk writes its slices; later chunks (and an accumulating call) add to them
  const bool first = c0 == 0 && !accumulate;
  if (kdev) cw = min(cw, 2 * *kdev);  // union columns: [hi | lo] of the K classes the device found
  constexpr int FR = G::FR, FC = G::FC, TR = G::kBR, TC = G::kBC;
  const int nMt = (M + TR - 1) / TR;
  const int nDt = (D + TC - 1) / TC;
  // Each XCD (a contiguous run of work ids) takes one block of a gm x (8 / gm) partition of
  // the frame x d tile grid: it reads dZ rows of its frame block and W columns of its d block
  const int work = xcd_swz(blockIdx.x, gridDim.x);
  const int s = work / (nMt * nDt);
  int mt, dt;
  block_tile(work % (nMt * nDt), nMt, nDt, gm, mt, dt);
  const int m0 = mt * TR, d0 = dt * TC;
  const int kb = s * slice;
  const int ke = min(cw, kb + slice);
  if (kb >= ke && !first) return;  // the first chunk writes every slice (zeros when empty)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // A: dZ rows (frames), k = vocabulary column; B: W_c viewed as rows d, k = vocabulary row
  const GOp A{dZ, chunk, M, cw, nullptr};
  const GOp B{W + static_cast<int64_t>(c0) * D, D, D, cw, nullptr};
  float* dst = part + static_cast<int64_t>(s) * M * D;
  // the accumulators start from this slice's partial sums of the earlier chunks (loaded
  // before the copy pipeline starts, so their latency hides behind its first copies)
  f32x16 acc[FR][FC];
#pragma unroll
  for (int i = 0; i < FR; ++i)
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      const int d = d0 + G::col_of(wave, lane, j);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + G::row_of(wave, lane, i, r);
        acc[i][j][r] = (first || d >= D || m >= M) ? 0.f : dst[static_cast<int64_t>(m) * D + d];
      }
    }
  // 8-wave tiles on the ping-pong schedule (each SIMD's two waves alternate products and copies)
  if constexpr (G::NW == 8) {
    G::template product<false>(A, B, m0, d0, kb, ke, acc);
  } else {
    PCTC_STAGES_G(G)
    G::template run<false>(A, B, m0, d0, kb, ke, st, acc);
  }
#pragma unroll
  for (int i = 0; i < FR; ++i)
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      const int d = d0 + G::col_of(wave, lane, j);
      if (d >= D) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + G::row_of(wave, lane, i, r);
        // rowscale (a first chunk only, whose partial sums start at zero): dZ rows were
        // written without their per-frame factor
        if (m < M) dst[static_cast<int64_t>(m) * D + d] = rowscale ? acc[i][j][r] * rowscale[m] : acc[i][j][r];
      }
    }
}

// One operand set of a dW product: out[(c0 + v) * D + d] = sum over frames of Z[m][v] Hs[m][d]
// for v < cw (cut to 2 *kdev when kdev is set: the union columns' [hi | lo] of the K classes
// the device found).  With nz > 1 the frames are split into nz slices of mslice frames and
// slice z writes its partial sums at out + z * zstride.
struct DwOp {
  const uint16_t* Z;
  int ld, c0, cw;
  float* out;
  int nz, mslice;
  int64_t zstride;
  const int32_t* kdev;
};

// dW products of up to two operand sets in one launch: work ids below tiles0 take P0's output
// tiles, the rest P1's (the union columns' dW_u in the last chunk's launch).
__global__ void __launch_bounds__(512, 1)
dw_gemm_bf16(DwOp P0, DwOp P1, int tiles0, const uint16_t* __restrict__ Hs, int M, int D) {
  using G = GDw;
  constexpr int FR = G::FR, FC = G::FC;
  PCTC_STAGES_G(G)
  const int work = xcd_swz(blockIdx.x, gridDim.x);
  const bool second = work >= tiles0;
  const DwOp P = second ? P1 : P0;
  const int w = second ? work - tiles0 : work;
  const int nDt = (D + kBC - 1) / kBC;
  int cw = P.cw;
  const int nVt = (cw + kBR - 1) / kBR;
  const int dt = w % nDt;
  const int vt = (w / nDt) % nVt;
  const int z = w / (nDt * nVt);
  const int v0 = vt * kBR, d0 = dt * kBC;
  const int mb = z * P.mslice;
  const int mlen = min(M - mb, P.mslice);
  if (P.kdev) cw = min(cw, 2 * *P.kdev);
  if (z >= P.nz || mlen <= 0 || v0 >= cw) return;
  float* const dW = P.out + static_cast<int64_t>(z) * P.zstride;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // A: Z viewed as rows v (columns of Z), k = frame; B: Hs viewed as rows d, k = frame
  const GOp A{P.Z + static_cast<int64_t>(mb) * P.ld, P.ld, cw, mlen, nullptr};
  const GOp B{Hs + static_cast<int64_t>(mb) * D, D, D, mlen, nullptr};
  f32x16 acc[FR][FC];
  G::run_pp(A, B, v0, d0, 0, mlen, st, acc);
#pragma unroll
  for (int i = 0; i < FR; ++i)
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      const int d = d0 + G::col_of(wave, lane, j);
      if (d >= D) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int v = v0 + G::row_of(wave, lane, i, r);
        if (v < cw) dW[static_cast<int64_t>(P.c0 + v) * D + d] = acc[i][j][r];
      }
    }
}

// Hs = H with the rows of excluded frames (g[m] == 0) set to zero.
__global__ void hs_build_bf16(const uint16_t* __restrict__ H, int64_t n, int D, const float* __restrict__ g,
                              uint16_t* __restrict__ Hs) {
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) * 8;
  if (i >= n) return;
  const int m = static_cast<int>(i / D);
  u32x4 v = *reinterpret_cast<const u32x4*>(H + i);
  if (g[m] == 0.f) v = u32x4{0u, 0u, 0u, 0u};
  *reinterpret_cast<u32x4*>(Hs + i) = v;
}

// Ht[d][m] = H[m][d] for m < M (zero where g is given and g[m] == 0), zero for m in [M, Mp); with
// Hs given, the same masked rows are also written there in H's layout (the hs_build_bf16 copy).
// 64 frames x 64 columns per workgroup through LDS, 16 bytes per access both ways (D is a
// multiple of 8, Mp of 64).
__global__ void __launch_bounds__(256) ht_build_bf16(const uint16_t* __restrict__ H, int M, int D,
                                                     const float* __restrict__ g, uint16_t* __restrict__ Hs,
                                                     uint16_t* __restrict__ Ht, int Mp) {
  __shared__ __attribute__((aligned(16))) uint16_t tile[64][72];  // rows 144 bytes apart
  const int m0 = blockIdx.x * 64, d0 = blockIdx.y * 64;
#pragma unroll
  for (int q = threadIdx.x; q < 512; q += 256) {  // 64 frames x 8 runs of 8 columns
    const int r = q >> 3, c = (q & 7) * 8;
    const int m = m0 + r, d = d0 + c;
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (m < M && d < D) {
      const int64_t i = static_cast<int64_t>(m) * D + d;
      if (!(g && g[m] == 0.f)) v = *reinterpret_cast<const u32x4*>(H + i);
      if (Hs) *reinterpret_cast<u32x4*>(Hs + i) = v;
    }
    *reinterpret_cast<u32x4*>(&tile[r][c]) = v;
  }
  __syncthreads();
#pragma unroll
  for (int q = threadIdx.x; q < 512; q += 256) {  // 64 columns x 8 runs of 8 frames
    const int r = q >> 3, c = (q & 7) * 8;
    const int d = d0 + r;
    if (d >= D) continue;
    u32x4 o;
#pragma unroll
    for (int k = 0; k < 4; ++k)
      o[k] = static_cast<uint32_t>(tile[c + 2 * k][r]) | (static_cast<uint32_t>(tile[c + 2 * k + 1][r]) << 16);
    *reinterpret_cast<u32x4*>(Ht + static_cast<int64_t>(d) * Mp + m0 + c) = o;
  }
}

// Hp = s_m Hs (bf16) for the dW product of the chunk whose dZ rows hold the normaliser's
// E = exp(z): its dense part is s_m E[m][v] with s_m = -g_m exp(-lambda_m) (rowscale, written
// by the finalize).  When the finalize's check failed (*einv: E unusable, the chunk is
// recomputed with its factor), Hp = Hs and rowscale = 1.
__global__ void hs_scale_bf16(const uint16_t* __restrict__ Hs, int64_t n, int D, const int32_t* __restrict__ einv,
                              float* __restrict__ rowscale, uint16_t* __restrict__ Hp) {
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) * 8;
  if (i >= n) return;
  const int m = static_cast<int>(i / D);
  const u32x4 v = *reinterpret_cast<const u32x4*>(Hs + i);
  if (*einv != 0) {
    if (i % D == 0) rowscale[m] = 1.f;  // no other thread reads it on this branch
    *reinterpret_cast<u32x4*>(Hp + i) = v;
    return;
  }
  const float sm = rowscale[m];
  u32x4 o;
#pragma unroll
  for (int k = 0; k < 4; ++k)
    o[k] = pack_bf16x2(bf16_to_f32(static_cast<uint16_t>(v[k] & 0xffffu)) * sm,
                       bf16_to_f32(static_cast<uint16_t>(v[k] >> 16)) * sm);
  *reinterpret_cast<u32x4*>(Hp + i) = o;
}

// ---------------------------------------------------------------------------------------
// Union-column part of the backward, computed beside the dense part -g p:
//   dH_u = G W_U,  dW_u = G^T Hs,  db_u = column sums of G
// (scatter_U(G) of Eq. vjp taken through the two products).  G is split into bf16 hi + lo
// halves laid side by side, Gb = [hi | lo] (K' = 2 ldK columns), so the matrix cores carry
// G to about 16 bits: dH_u is one product against [W_U; W_U], dW_u two row blocks that are
// summed when merged into dW.
// ---------------------------------------------------------------------------------------
// Gb [M][2 ldK]: columns j and K + j hold the hi and lo halves of G[m][j] for j < K (K the
// union size found on the device, <= ldK) and the columns from 2K on hold zeros (a product's
// copy of a k-run may reach past 2K; those values meet zero rows of W_U, and must be finite).
__global__ void __launch_bounds__(256)
union_split_bf16(const float* __restrict__ G, int ldG, const int32_t* __restrict__ Kdev, int ldK, int M,
                 uint16_t* __restrict__ Gb) {
  const int K = *Kdev;
  const int64_t n = static_cast<int64_t>(M) * ldK;
  // a few hundred workgroups stride over the elements: the launch runs beside a recompute,
  // whose compute units it should not churn with thousands of tiny workgroups
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    const int m = static_cast<int>(i / ldK), j = static_cast<int>(i % ldK);
    const float* grow = G + static_cast<int64_t>(m) * ldG;
    uint16_t* row = Gb + static_cast<int64_t>(m) * (2 * ldK);
#pragma unroll
    for (int h = 0; h < 2; ++h) {  // columns j and ldK + j
      const int c = j + h * ldK;
      uint16_t out = 0;
      if (c < K) {
        out = f32_to_bf16(grow[c]);
      } else if (c < 2 * K) {
        const float x = grow[c - K];
        out = f32_to_bf16(x - bf16_to_f32(f32_to_bf16(x)));
      }
      row[c] = out;
    }
  }
}

// WU2 [2 ldK][D]: rows j and K + j hold W[U_j] for j < K; the rows past 2K are never read.
__global__ void __launch_bounds__(256)
union_rows_bf16(const uint16_t* __restrict__ W, int D, const int32_t* __restrict__ u_ids,
                const int32_t* __restrict__ Kdev, uint16_t* __restrict__ WU2) {
  const int K = *Kdev;
  for (int r = blockIdx.x; r < 2 * K; r += gridDim.x) {
    const int j = r < K ? r : r - K;
    const uint16_t* src = W + static_cast<int64_t>(u_ids[j]) * D;
    for (int d = threadIdx.x * 8; d < D; d += 256 * 8)
      *reinterpret_cast<u32x4*>(WU2 + static_cast<int64_t>(r) * D + d) = *reinterpret_cast<const u32x4*>(src + d);
  }
}

// dbp[z][j] = sum of G[m][j] over the frames of slice z (fp32, in frame order)
__global__ void __launch_bounds__(256)
union_colsum_bf16(const float* __restrict__ G, int ldG, int M, int K_max, int mper, float* __restrict__ dbp) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  const int z = blockIdx.y;
  if (j >= K_max) return;
  const int mb = z * mper, me = min(M, mb + mper);
  float acc = 0.f;
  for (int m = mb; m < me; ++m) acc += G[static_cast<int64_t>(m) * ldG + j];
  dbp[static_cast<int64_t>(z) * K_max + j] = acc;
}

// dW[U_j, :] += sum over the frame slices of dW_u2[j, :] + dW_u2[K + j, :];
// db[U_j] += sum_z dbp[z][j]
__global__ void __launch_bounds__(256)
union_merge_bf16(const int32_t* __restrict__ Kdev, const int32_t* __restrict__ u_ids, int D, int ldK, int K_max,
                 int nz, int nzw, const float* __restrict__ dWu2, const float* __restrict__ dbp, float* __restrict__ dW,
                 float* __restrict__ db) {
  const int j = blockIdx.y;
  if (j >= *Kdev) return;
  const int v = u_ids[j];
  const int d = blockIdx.x * 256 + threadIdx.x;
  if (dW && d < D) {
    const int K = *Kdev;
    float s = 0.f;
    for (int z = 0; z < nzw; ++z) {
      const float* p = dWu2 + static_cast<int64_t>(z) * 2 * ldK * D;
      s += p[static_cast<int64_t>(j) * D + d] + p[static_cast<int64_t>(K + j) * D + d];
    }
    dW[static_cast<int64_t>(v) * D + d] += s;
  }
  if (db && blockIdx.x == 0 && threadIdx.x == 0) {
    float s = 0.f;
    for (int z = 0; z < nz; ++z) s += dbp[static_cast<int64_t>(z) * K_max + j];
    db[v] += s;
  }
}

namespace {
constexpr int kColSlices = 16;
struct UnionCorrLayout {
  int ldK, nz, mslice;  // dW_u over nz slices of mslice frames (one: every frame)
  size_t o_dwu, o_wu, o_dbp, total;
};
// [dW_u (only when dW is wanted)][W_U rows twice][db_u slices]; the [hi | lo] copy of G lives
// outside (gb_bytes, in the region of S, which is dead once the lattice is done).  dW_u is one
// launch's worth of 256 x 256 tiles over all frames, like a dense dW tile, so that it can ride
// in the last round of the last chunk's dense dW launch.
UnionCorrLayout union_corr_layout(int M, int D, int K_max, bool want_dW) {
  UnionCorrLayout L;
  L.ldK = (K_max + 7) / 8 * 8;
  const size_t k2 = static_cast<size_t>(2) * L.ldK;
  L.nz = 1;
  L.mslice = M > 0 ? M : 1;
  L.o_dwu = 0;
  L.o_wu = L.o_dwu + (want_dW ? align_up(static_cast<size_t>(L.nz) * k2 * D * sizeof(float), 256) : 0);
  L.o_dbp = L.o_wu + align_up(k2 * D * sizeof(uint16_t), 256);
  L.total = L.o_dbp + align_up(static_cast<size_t>(kColSlices) * K_max * sizeof(float), 256);
  return L;
}
}  // namespace

size_t union_corr_bytes(int M, int D, int K_max, bool want_dW) {
  return union_corr_layout(M, D, K_max, want_dW).total;
}
size_t union_gb_bytes(int M, int K_max) {
  return static_cast<size_t>(M) * 2 * ((K_max + 7) / 8 * 8) * sizeof(uint16_t);
}

DwExtra union_dw_extra(int M, int D, int K_max, const int32_t* Kdev, void* scratch, const uint16_t* Gb) {
  DwExtra x;
  if (M <= 0 || K_max <= 0) return x;
  const UnionCorrLayout L = union_corr_layout(M, D, K_max, true);
  x.Z = Gb;
  x.ld = 2 * L.ldK;
  x.cols = 2 * L.ldK;
  x.kdev = Kdev;
  x.out = reinterpret_cast<float*>(static_cast<char*>(scratch) + L.o_dwu);
  return x;
}

hipError_t launch_union_part_bf16(const float* G, int ldG, const int32_t* Kdev, int K_max, const int32_t* u_ids,
                                  const uint16_t* W, const uint16_t* Hs, int M, int D, float* dH, bool dh_later,
                                  bool want_dW, bool want_db, void* scratch, uint16_t* Gb, hipStream_t stream,
                                  bool dw_elsewhere) {
  const bool want_dH = dH != nullptr || dh_later;
  if (M <= 0 || K_max <= 0) return hipSuccess;
  if (want_dW && !Hs) return hipErrorInvalidValue;
  const UnionCorrLayout L = union_corr_layout(M, D, K_max, want_dW);
  char* sc = static_cast<char*>(scratch);
  const int k2 = 2 * L.ldK;
  if (want_dH || want_dW) {
    Prof pr("union_prep", stream);
    const int64_t n = static_cast<int64_t>(M) * L.ldK;
    const int64_t blocks = (n + 255) / 256;
    hipLaunchKernelGGL(union_split_bf16, dim3(static_cast<unsigned>(blocks < 512 ? blocks : 512)), dim3(256), 0,
                       stream, G, ldG, Kdev, L.ldK, M, Gb);
  }
  if (want_dH) {
    uint16_t* WU2 = reinterpret_cast<uint16_t*>(sc + L.o_wu);
    hipLaunchKernelGGL(union_rows_bf16, dim3(k2 < 256 ? k2 : 256), dim3(256), 0, stream, W, D, u_ids, Kdev, WU2);
    if (!dh_later) {
      const int tiles = ((M + GUh::kBR - 1) / GUh::kBR) * ((D + GUh::kBC - 1) / GUh::kBC);
      Prof pr("union_dh", stream);
      hipLaunchKernelGGL((dh_gemm_bf16<GUh, 2>), dim3(tiles), dim3(GUh::kThreads), 0, stream, Gb, M, k2, WU2, D, 0,
                         k2, k2, dH, dh_xcd_rows(M, D), 0, Kdev, nullptr);
    }
  }
  if (want_dW && !dw_elsewhere) {
    const int tiles = ((k2 + kBR - 1) / kBR) * ((D + kBC - 1) / kBC) * L.nz;
    const DwOp p{Gb, k2, 0, k2, reinterpret_cast<float*>(sc + L.o_dwu), L.nz, L.mslice,
                 static_cast<int64_t>(k2) * D, Kdev};
    Prof pr("union_dw", stream);
    hipLaunchKernelGGL(dw_gemm_bf16, dim3(tiles), dim3(GDw::kThreads), 0, stream, p, p, tiles, Hs, M, D);
  }
  if (want_db) {
    const int mper = (M + kColSlices - 1) / kColSlices;
    Prof pr("union_colsum", stream);
    hipLaunchKernelGGL(union_colsum_bf16, dim3((K_max + 255) / 256, kColSlices), dim3(256), 0, stream, G, ldG, M,
                       K_max, mper, reinterpret_cast<float*>(sc + L.o_dbp));
  }
  return hipGetLastError();
}

hipError_t launch_union_dh_bf16(const uint16_t* Gb, const int32_t* Kdev, int K_max, int M, int D, float* dH,
                                void* scratch, bool want_dW, hipStream_t stream) {
  if (M <= 0 || K_max <= 0 || !dH) return hipSuccess;
  const UnionCorrLayout L = union_corr_layout(M, D, K_max, want_dW);
  const int k2 = 2 * L.ldK;
  const uint16_t* WU2 = reinterpret_cast<const uint16_t*>(static_cast<char*>(scratch) + L.o_wu);
  const int tiles = ((M + GUh::kBR - 1) / GUh::kBR) * ((D + GUh::kBC - 1) / GUh::kBC);
  Prof pr("union_dh", stream);
  hipLaunchKernelGGL((dh_gemm_bf16<GUh, 2>), dim3(tiles), dim3(GUh::kThreads), 0, stream, Gb, M, k2, WU2, D, 0, k2,
                     k2, dH, dh_xcd_rows(M, D), 1, Kdev, nullptr);
  return hipGetLastError();
}

hipError_t launch_union_merge_bf16(const int32_t* Kdev, int K_max, const int32_t* u_ids, int M, int D, float* dW,
                                   float* db, void* scratch, hipStream_t stream) {
  if (M <= 0 || K_max <= 0 || (!dW && !db)) return hipSuccess;
  const UnionCorrLayout L = union_corr_layout(M, D, K_max, dW != nullptr);
  char* sc = static_cast<char*>(scratch);
  Prof pr("union_merge", stream);
  hipLaunchKernelGGL(union_merge_bf16, dim3((D + 255) / 256, K_max), dim3(256), 0, stream, Kdev, u_ids, D, L.ldK,
                     K_max, kColSlices, L.nz, reinterpret_cast<const float*>(sc + L.o_dwu),
                     reinterpret_cast<const float*>(sc + L.o_dbp), dW, db);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// launchers (bf16 path)
// ---------------------------------------------------------------------------------------

// Vocabulary split of a normaliser or argmax launch: each workgroup takes a run of vper / 256
// vocabulary tiles for one frame tile (partition p covers rows [p vper, (p + 1) vper)).  Wide
// heads: one tile per workgroup while the partitions fit the partial buffer (the long k
// loop makes a workgroup's start-up cost small; shorter runs also spread the last tiles
// better).  Narrow heads: the fewest runs within 256 partitions, so that each workgroup's
// copy pipeline runs through several tiles.  (Runs chosen to fill the last round of
// workgroups evenly measured slower for narrow heads: the run length also sets the L2 reuse
// of the tile order.)
struct LseSplit {
  bool wide;  // D >= kWideD: one vocabulary tile per partition (argmax: GWide tiles)
  int vper, P, nM;
};

static LseSplit lse_split_bf16(int M, int D, int V) {
  LseSplit s;
  s.wide = D >= kWideD;
  constexpr int TR = 256, TC = 256;
  static_assert(GWide::kBR == TR && GWide::kBC == TC && GMid::kBR == TR && GMid::kBC == TC, "tile shapes");
  const int vtiles = (V + TR - 1) / TR;
  s.nM = (M + TC - 1) / TC;
  const int maxp = lse_max_parts(D);
  int run = (vtiles + maxp - 1) / maxp;
  if (!s.wide && run < kMidRun) run = kMidRun;
  s.vper = run * TR;
  s.P = (V + s.vper - 1) / s.vper;
  return s;
}

hipError_t launch_lse_partial_bf16(const uint16_t* H, int M, int D, const uint16_t* W, const float* bias, int V,
                                   float2* partials, int* P_out, hipStream_t stream) {
  const LseSplit sp = lse_split_bf16(M, D, V);
  const int vper = sp.vper, Peff = sp.P;
  *P_out = Peff;
  Prof pr("lse_partial", stream);
  const size_t bsh = bias ? static_cast<size_t>(vper) * sizeof(float) : 0;
  // every head on the 32-deep four-stage tiles (for wide heads each vocabulary tile is its own
  // partition; the 64-deep two-stage tiles measured 4% slower there)
  const dim3 grid(sp.nM * Peff);
  if (bias) {
    hipLaunchKernelGGL((lse_partial_bf16<GMid, true, 1>), grid, dim3(GMid::kThreads), bsh, stream, H, M, D, W, bias,
                       V, Peff, vper, partials);
  } else {
    hipLaunchKernelGGL((lse_partial_bf16<GMid, false, 1>), grid, dim3(GMid::kThreads), 0, stream, H, M, D, W, bias,
                       V, Peff, vper, partials);
  }
  return hipGetLastError();
}

hipError_t launch_amax_partial_bf16(const uint16_t* H, int M, int D, const uint16_t* W, const float* bias, int V,
                                    float2* partials, int* P_out, hipStream_t stream) {
  const LseSplit sp = lse_split_bf16(M, D, V);
  const int vper = sp.vper, Peff = sp.P;
  *P_out = Peff;
  Prof pr("amax_partial", stream);
  const size_t bsh = bias ? static_cast<size_t>(vper) * sizeof(float) : 0;
  const dim3 grid(grouped_grid(sp.nM, Peff));
  if (sp.wide) {
    if (bias)
      hipLaunchKernelGGL((amax_partial_bf16<GWide, true, 1>), grid, dim3(GWide::kThreads), bsh, stream, H, M, D, W,
                         bias, V, Peff, vper, partials);
    else
      hipLaunchKernelGGL((amax_partial_bf16<GWide, false, 1>), grid, dim3(GWide::kThreads), 0, stream, H, M, D, W,
                         bias, V, Peff, vper, partials);
  } else if (bias) {
    hipLaunchKernelGGL((amax_partial_bf16<GMid, true, 1>), grid, dim3(GMid::kThreads), bsh, stream, H, M, D, W, bias,
                       V, Peff, vper, partials);
  } else {
    hipLaunchKernelGGL((amax_partial_bf16<GMid, false, 1>), grid, dim3(GMid::kThreads), 0, stream, H, M, D, W, bias,
                       V, Peff, vper, partials);
  }
  return hipGetLastError();
}

hipError_t launch_gather_s_bf16(const uint16_t* H, int M, int D, const uint16_t* W, const float* bias,
                                const int32_t* u_ids, const int32_t* K, int K_max, const double* lam, float* S, int ldS,
                                hipStream_t stream, double* Zd) {
  const int nMt = (M + kFC - 1) / kFC;
  const int nJt = (K_max + kFR - 1) / kFR;
  Prof pr("gather_s", stream);
  hipLaunchKernelGGL(gather_s_bf16, dim3(nMt * nJt), dim3(GFwd::kThreads), 0, stream, H, M, D, W, bias, u_ids, K, lam,
                     S, ldS, Zd);
  return hipGetLastError();
}

hipError_t launch_bwd_chunk_bf16(const uint16_t* Hs, int M, int D, const uint16_t* W, const float* bias, int c0,
                                 int cw, const float2* lam2, const float* G, int ldG, const float* g,
                                 const int32_t* remap, const float* S, int ldS, uint16_t* dZ, int chunk, float* part,
                                 int slice, bool recompute, bool want_dH, bool want_dW, float* dW, float* db,
                                 float* dbpart, hipStream_t stream, const DwExtra* extra, const ChunkE* ce,
                                 const uint16_t* Hst, int Mp) {
  // wide heads: one 8-wave 256 x 256 workgroup per CU (the long k loop hides the epilogue);
  // narrow heads: two 4-wave 256 x 128 workgroups per CU, so that one's epilogue (exp, pack,
  // staged stores: VALU-bound) overlaps the other's products
  const bool wide = D >= kWideD;
  const int nMt = (M + (wide ? GWide::kBC : GFwd::kBC) - 1) / (wide ? GWide::kBC : GFwd::kBC);
  if (recompute) {
    const int nVt = (cw + kFR - 1) / kFR;
    const dim3 grid(grouped_grid(nMt, nVt));
    // with ce the launch only recomputes when the normaliser's rows are unusable
    Prof pr(ce ? "recompute_check" : "recompute_dz", stream);
#define PCTC_RECOMPUTE(GC, OCC, BI, DBI)                                                                             \
  hipLaunchKernelGGL((recompute_dz_bf16<GC, BI, DBI, OCC>), grid, dim3(GC::kThreads), 0, stream, Hs, M, D, W, bias, \
                     c0, cw, lam2, g, remap, S, ldS, G, ldG, dZ, chunk, dbpart)
#define PCTC_RECOMPUTE_CFG(GC, OCC)           \
  if (bias) {                                 \
    if (db) PCTC_RECOMPUTE(GC, OCC, true, true);  \
    else PCTC_RECOMPUTE(GC, OCC, true, false);    \
  } else {                                    \
    if (db) PCTC_RECOMPUTE(GC, OCC, false, true); \
    else PCTC_RECOMPUTE(GC, OCC, false, false);   \
  }
    if (!ce && wide) {
      PCTC_RECOMPUTE_CFG(GWide, 1)
    } else if (ce || (!bias && !db && !remap && D % (GMid::kNS * GMid::KK * 16) == 0)) {
      // one round of workgroups (one per CU, 256 x 256 tiles), each taking a run of vocabulary
      // tiles for one frame tile; kRcCus workgroups at most, so that the second stream's
      // lattice and union work keeps a few CUs of every XCD beside them
      const int nMt2 = (M + GMid::kBC - 1) / GMid::kBC;
      const int runs = max(1, min(nVt, kRcCus / nMt2));
      const int run = (nVt + runs - 1) / runs;
      const int nruns = (nVt + run - 1) / run;
      if (Hst)
        hipLaunchKernelGGL(recompute_run_bf16<true>, dim3(nMt2 * nruns), dim3(GMid::kThreads), 0, stream, Hs, Hst,
                           Mp, M, D, W, c0, cw, run, lam2, g, dZ, chunk, ce ? ce->einv : nullptr);
      else
        hipLaunchKernelGGL(recompute_run_bf16<false>, dim3(nMt2 * nruns), dim3(GMid::kThreads), 0, stream, Hs, Hst,
                           Mp, M, D, W, c0, cw, run, lam2, g, dZ, chunk, ce ? ce->einv : nullptr);
    } else {
      PCTC_RECOMPUTE_CFG(GFwd, 2)
    }
#undef PCTC_RECOMPUTE_CFG
#undef PCTC_RECOMPUTE
  }
  if (db && recompute) {
    Prof pr("db_reduce", stream);
    hipLaunchKernelGGL(db_reduce_bf16, dim3((cw + 255) / 256), dim3(256), 0, stream, dbpart, nMt, chunk, cw, db + c0);
  }
  if (want_dH) {
    const int tiles = ((M + kBR - 1) / kBR) * ((D + kBC - 1) / kBC);
    const int ns = (cw + slice - 1) / slice;
    Prof pr("dh_gemm", stream);
    hipLaunchKernelGGL((dh_gemm_bf16<GDh, 1>), dim3(tiles * ns), dim3(GDh::kThreads), 0, stream, dZ, M, chunk, W, D,
                       c0, cw, slice, part, dh_xcd_rows(M, D), 0, nullptr, ce ? ce->rowscale : nullptr);
  }
  if (want_dW) {
    const int nDt = (D + kBC - 1) / kBC;
    const int tiles0 = ((cw + kBR - 1) / kBR) * nDt;
    const DwOp p0{dZ, chunk, c0, cw, dW, 1, M, 0, nullptr};
    DwOp p1 = p0;
    int tiles1 = 0;
    if (extra && extra->Z) {  // the union columns' dW_u, in this launch's last round
      p1 = DwOp{extra->Z, extra->ld, 0, extra->cols, extra->out, 1, M, 0, extra->kdev};
      tiles1 = ((extra->cols + kBR - 1) / kBR) * nDt;
    }
    Prof pr("dw_gemm", stream);
    hipLaunchKernelGGL(dw_gemm_bf16, dim3(tiles0 + tiles1), dim3(GDw::kThreads), 0, stream, p0, p1, tiles0,
                       ce ? ce->Hp : Hs, M, D);
  }
  return hipGetLastError();
}

hipError_t launch_hs_scale_bf16(const uint16_t* Hs, int M, int D, const int32_t* einv, float* rowscale, uint16_t* Hp,
                                hipStream_t stream) {
  const int64_t n = static_cast<int64_t>(M) * D;
  const int64_t threads = (n + 7) / 8;
  if (threads <= 0) return hipSuccess;
  Prof pr("hs_scale", stream);
  hipLaunchKernelGGL(hs_scale_bf16, dim3(static_cast<unsigned>((threads + 255) / 256)), dim3(256), 0, stream, Hs, n, D,
                     einv, rowscale, Hp);
  return hipGetLastError();
}

int lse_e_parts_bf16(int M, int D, int V, int chunk) {
  if (M <= 0 || D % (GMid::kNS * GMid::KK * 16) != 0 || chunk <= 0) return 0;
  const LseSplit sp = lse_split_bf16(M, D, V);
  if (chunk % sp.vper != 0) return 0;
  const int ep = chunk / sp.vper;
  return ep < sp.P ? ep : sp.P;
}

hipError_t launch_lse_partial_e_bf16(const uint16_t* H, int M, int D, const uint16_t* W, int V, float2* partials,
                                     int* P_out, uint16_t* E, int epitch, int eparts, int32_t* einv,
                                     hipStream_t stream, const uint16_t* Ht, int Mp) {
  const LseSplit sp = lse_split_bf16(M, D, V);
  *P_out = sp.P;
  Prof pr("lse_partial", stream);
  if (Ht)
    hipLaunchKernelGGL(lse_partial_e_bf16<true>, dim3(sp.nM * sp.P), dim3(GMid::kThreads), 0, stream, H, Ht, Mp, M, D,
                       W, V, sp.P, sp.vper, partials, E, epitch, eparts, einv);
  else
    hipLaunchKernelGGL(lse_partial_e_bf16<false>, dim3(sp.nM * sp.P), dim3(GMid::kThreads), 0, stream, H, Ht, Mp, M,
                       D, W, V, sp.P, sp.vper, partials, E, epitch, eparts, einv);
  return hipGetLastError();
}

hipError_t launch_ht_build_bf16(const uint16_t* H, int M, int D, const float* g, uint16_t* Hs, uint16_t* Ht, int Mp,
                                hipStream_t stream) {
  if (M <= 0) return hipSuccess;
  Prof pr(Hs ? "hs_build" : "ht_build", stream);
  hipLaunchKernelGGL(ht_build_bf16, dim3(static_cast<unsigned>(Mp / 64), static_cast<unsigned>((D + 63) / 64)),
                     dim3(256), 0, stream, H, M, D, g, Hs, Ht, Mp);
  return hipGetLastError();
}

hipError_t launch_hs_build_bf16(const uint16_t* H, int M, int D, const float* g, uint16_t* Hs, hipStream_t stream) {
  const int64_t n = static_cast<int64_t>(M) * D;
  const int64_t threads = (n + 7) / 8;
  Prof pr("hs_build", stream);
  hipLaunchKernelGGL(hs_build_bf16, dim3(static_cast<unsigned>((threads + 255) / 256)), dim3(256), 0, stream, H, n,
                     D, g, Hs);
  return hipGetLastError();
}

}  // namespace pctc
