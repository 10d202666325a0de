// Device-side building blocks shared by the Pruned CTC kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pctc {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr double kLog2eD = 1.4426950408889634074;
constexpr double kLn2D = 0.69314718055994530942;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round-to-nearest-even float -> bf16 bits (NaN kept quiet).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x7fffffu)) return static_cast<uint16_t>((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Two floats rounded to bfloat16 (nearest even) and packed, the first in the low half.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __attribute__((ext_vector_type(2))) float f2_;
  typedef __attribute__((ext_vector_type(2))) __bf16 b2_;
  const b2_ b = __builtin_convertvector(f2_{lo, hi}, b2_);
  return __builtin_bit_cast(uint32_t, b);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// Value of lane (l ^ 32): the other half of the wavefront.
__device__ __forceinline__ float swap_halves(float x) {
  return __shfl_xor(x, 32, 64);
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// ---------------------------------------------------------------------------------------
// Matrix-core tile engine.
//
// C[i][j] = sum_k A[i][k] * B[j][k] for a BR x BC output tile, where A supplies BR rows
// and B supplies BC rows, both indexed by the contraction index k.  Both operands are
// staged through LDS as [row][k] (k contiguous, padded pitch) and consumed by
// 32x32 matrix-core instructions:
//   bf16: v_mfma_f32_32x32x16_bf16 -- per lane 8 bf16 of A and of B per instruction;
//   f32:  v_mfma_f32_32x32x2_f32  -- per lane 1 float of A and of B per instruction.
// Within each 16-wide k step, lane half h = lane/32 always carries k in [8h, 8h+8)
// (bf16: one instruction; f32: eight instructions, the e-th using k = 8h + e).  A and B
// use the same assignment, so every k is paired exactly once.
// Accumulator layout of a 32x32 block (16 floats per lane): lane l holds column
// j = l % 32 and rows i = 8*(r/4) + 4*(l/32) + (r%4) for register r.
// Four wavefronts tile the output 2 x 2; each wavefront owns (BR/2) x (BC/2), i.e.
// FR x FC blocks of 32x32.
// ---------------------------------------------------------------------------------------

template <typename T>
struct ElemTraits;
template <>
struct ElemTraits<uint16_t> {  // bf16 bits
  static constexpr int kVec = 8;  // elements per 16-byte vector
};
template <>
struct ElemTraits<float> {
  static constexpr int kVec = 4;
};

// How an operand is laid out in global memory.
//  KMajor:  element (row r, k) at base[r * pitch + k]        (k contiguous)
//  RowMajorT: element (row r, k) at base[k * pitch + r]      (rows contiguous)
//  Gathered: element (row r, k) at base[rows[r] * pitch + k] (k contiguous, row table)
enum class Lay { KMajor, RowMajorT, Gathered };

template <typename T>
struct Operand {
  const T* base;
  int64_t pitch;    // elements
  int rows;         // valid rows (rows beyond read as zero)
  int kmax;         // valid k (k beyond read as zero)
  const int* rowidx;  // Gathered only
  const int* rowcount;  // Gathered only: device scalar limiting valid rows (may be null)
};

template <typename T, int BR, int BC, int BK>
struct TileShape {
  static constexpr int kVec = ElemTraits<T>::kVec;
  static constexpr int kPad = (sizeof(T) == 2) ? 8 : 4;  // 16 bytes of padding per row
  static constexpr int kPitch = BK + kPad;              // LDS row pitch in elements
  static constexpr int kLdsA = BR * kPitch;
  static constexpr int kLdsB = BC * kPitch;
  static constexpr int kLdsElems = kLdsA + kLdsB;
  static constexpr int FR = BR / 64;  // 32x32 blocks per wave along rows
  static constexpr int FC = BC / 64;  // 32x32 blocks per wave along columns
};

// Per-thread register staging of one operand tile (global -> registers -> LDS).
template <typename T, Lay L, int NR, int BK>
struct TileLoader {
  static constexpr int kVec = ElemTraits<T>::kVec;
  // KMajor / Gathered: NR rows x BK k, each thread loads whole 16-byte k-vectors.
  // RowMajorT: NR rows x BK k, each thread loads 16-byte row-vectors at 4 consecutive k
  //            (bf16: 8 rows x 4 k block) and transposes them in registers.
  static constexpr int kVecs = (NR * BK) / kVec;        // 16-byte vectors per tile
  static constexpr int kPerThread = kVecs / 256;
  static_assert(kVecs % 256 == 0, "tile must split evenly over 256 threads");
  u32x4 r[kPerThread];

  __device__ __forceinline__ void load(const Operand<T>& op, int row0, int k0, int tid) {
    if constexpr (L == Lay::KMajor || L == Lay::Gathered) {
      constexpr int kvecs_per_row = BK / kVec;
      int nvalid = op.rows;
      if constexpr (L == Lay::Gathered) {
        if (op.rowcount) nvalid = min(nvalid, *op.rowcount);
      }
#pragma unroll
      for (int p = 0; p < kPerThread; ++p) {
        int idx = tid + 256 * p;
        int rr = idx / kvecs_per_row;
        int kv = idx % kvecs_per_row;
        int row = row0 + rr;
        int k = k0 + kv * kVec;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (row < nvalid && k < op.kmax) {
          int64_t grow = row;
          if constexpr (L == Lay::Gathered) grow = op.rowidx[row];
          v = *reinterpret_cast<const u32x4*>(op.base + grow * op.pitch + k);
        }
        r[p] = v;
      }
    } else {
      // RowMajorT: vector = kVec consecutive rows at one k.  Thread block = kVec rows x 4 k.
      constexpr int rgroups = NR / kVec;
      constexpr int kgroups = BK / 4;
      static_assert(rgroups * kgroups == 256 * (kPerThread / 4), "layout");
#pragma unroll
      for (int p = 0; p < kPerThread / 4; ++p) {
        int blk = tid + 256 * p;
        int rg = blk % rgroups;
        int kg = blk / rgroups;
        int row = row0 + rg * kVec;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          int k = k0 + kg * 4 + kk;
          u32x4 v = {0u, 0u, 0u, 0u};
          if (k < op.kmax && row < op.rows) {
            v = *reinterpret_cast<const u32x4*>(op.base + static_cast<int64_t>(k) * op.pitch + row);
          }
          r[p * 4 + kk] = v;
        }
      }
    }
  }

  __device__ __forceinline__ void store(T* lds, int tid) const {
    using Shape = TileShape<T, 64, 64, BK>;
    constexpr int pitch = Shape::kPitch;
    if constexpr (L == Lay::KMajor || L == Lay::Gathered) {
      constexpr int kvecs_per_row = BK / kVec;
#pragma unroll
      for (int p = 0; p < kPerThread; ++p) {
        int idx = tid + 256 * p;
        int rr = idx / kvecs_per_row;
        int kv = idx % kvecs_per_row;
        *reinterpret_cast<u32x4*>(lds + rr * pitch + kv * kVec) = r[p];
      }
    } else {
      constexpr int rgroups = NR / kVec;
#pragma unroll
      for (int p = 0; p < kPerThread / 4; ++p) {
        int blk = tid + 256 * p;
        int rg = blk % rgroups;
        int kg = blk / rgroups;
        if constexpr (sizeof(T) == 2) {
          // r[p*4+kk].dword[q] holds rows (2q, 2q+1) at k = kg*4+kk.
          // Output row i (0..7): 4 bf16 at k = kg*4 .. kg*4+3 -> two dwords.
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const int q = i >> 1;
            const uint32_t sel = (i & 1) ? 0x07060302u : 0x05040100u;
            uint32_t d0 = __builtin_amdgcn_perm(r[p * 4 + 1][q], r[p * 4 + 0][q], sel);
            uint32_t d1 = __builtin_amdgcn_perm(r[p * 4 + 3][q], r[p * 4 + 2][q], sel);
            u32x2 w = {d0, d1};
            *reinterpret_cast<u32x2*>(lds + (rg * 8 + i) * pitch + kg * 4) = w;
          }
        } else {
          // r[p*4+kk][i] is row i at k = kg*4+kk; output row i = 4 consecutive k.
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            u32x4 w = {r[p * 4 + 0][i], r[p * 4 + 1][i], r[p * 4 + 2][i], r[p * 4 + 3][i]};
            *reinterpret_cast<u32x4*>(lds + (rg * 4 + i) * pitch + kg * 4) = w;
          }
        }
      }
    }
  }
};

// Fragment multiply of one 16-wide k step for a wave's FR x FC blocks.
template <typename T, int FR, int FC, int PITCH>
__device__ __forceinline__ void mma_k16(const T* ldsA, const T* ldsB, int wrow0, int wcol0, int kk,
                                        int lane, f32x16 (&acc)[FR][FC]) {
  const int lr = lane & 31;
  const int lh = lane >> 5;
  if constexpr (sizeof(T) == 2) {
    bf16x8 a[FR], b[FC];
#pragma unroll
    for (int i = 0; i < FR; ++i)
      a[i] = *reinterpret_cast<const bf16x8*>(ldsA + (wrow0 + 32 * i + lr) * PITCH + kk + 8 * lh);
#pragma unroll
    for (int j = 0; j < FC; ++j)
      b[j] = *reinterpret_cast<const bf16x8*>(ldsB + (wcol0 + 32 * j + lr) * PITCH + kk + 8 * lh);
#pragma unroll
    for (int i = 0; i < FR; ++i)
#pragma unroll
      for (int j = 0; j < FC; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
  } else {
    typedef __attribute__((ext_vector_type(4))) float f32x4;
    f32x4 a[FR][2], b[FC][2];
#pragma unroll
    for (int i = 0; i < FR; ++i) {
      const float* pa = ldsA + (wrow0 + 32 * i + lr) * PITCH + kk + 8 * lh;
      a[i][0] = *reinterpret_cast<const f32x4*>(pa);
      a[i][1] = *reinterpret_cast<const f32x4*>(pa + 4);
    }
#pragma unroll
    for (int j = 0; j < FC; ++j) {
      const float* pb = ldsB + (wcol0 + 32 * j + lr) * PITCH + kk + 8 * lh;
      b[j][0] = *reinterpret_cast<const f32x4*>(pb);
      b[j][1] = *reinterpret_cast<const f32x4*>(pb + 4);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int i = 0; i < FR; ++i)
#pragma unroll
        for (int j = 0; j < FC; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][e >> 2][e & 3], b[j][e >> 2][e & 3],
                                                          acc[i][j], 0, 0, 0);
  }
}

// One BR x BC tile: C = A[row0:row0+BR, 0:K] . B[col0:col0+BC, 0:K]^T into acc.
// LDS single buffer with register prefetch of the next k tile.  Caller provides
// LDS of TileShape::kLdsElems elements.  All 256 threads must call.
template <typename T, int BR, int BC, int BK, Lay LA, Lay LB>
__device__ __forceinline__ void tile_gemm(const Operand<T>& A, const Operand<T>& B, int row0, int col0,
                                          int kbegin, int kend, T* lds,
                                          f32x16 (&acc)[BR / 64][BC / 64]) {
  using Shape = TileShape<T, BR, BC, BK>;
  constexpr int FR = Shape::FR, FC = Shape::FC, PITCH = Shape::kPitch;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wrow0 = (wave >> 1) * (BR / 2);
  const int wcol0 = (wave & 1) * (BC / 2);
  T* ldsA = lds;
  T* ldsB = lds + Shape::kLdsA;
#pragma unroll
  for (int i = 0; i < FR; ++i)
#pragma unroll
    for (int j = 0; j < FC; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  TileLoader<T, LA, BR, BK> la;
  TileLoader<T, LB, BC, BK> lb;
  if (kbegin >= kend) return;
  la.load(A, row0, kbegin, tid);
  lb.load(B, col0, kbegin, tid);
  for (int k0 = kbegin; k0 < kend; k0 += BK) {
    __syncthreads();
    la.store(ldsA, tid);
    lb.store(ldsB, tid);
    __syncthreads();
    if (k0 + BK < kend) {
      la.load(A, row0, k0 + BK, tid);
      lb.load(B, col0, k0 + BK, tid);
    }
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) mma_k16<T, FR, FC, PITCH>(ldsA, ldsB, wrow0, wcol0, kk, lane, acc);
  }
}

// Row index (within the tile) of accumulator register r of block (i, .) for this lane.
template <int BR>
__device__ __forceinline__ int acc_row(int wave, int lane, int i, int r) {
  return (wave >> 1) * (BR / 2) + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}
template <int BC>
__device__ __forceinline__ int acc_col(int wave, int lane, int j) {
  return (wave & 1) * (BC / 2) + 32 * j + (lane & 31);
}

}  // namespace pctc
