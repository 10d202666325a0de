// bf16 matrix-core tile engine for gfx950 with direct global->LDS staging.
//
// C[i][j] = sum_k A[i][k] B[j][k] over one BR x BC tile (4 wavefronts, 2 x 2; each owns
// (BR/2) x (BC/2) = FR x FC blocks of 32x32 accumulated by v_mfma_f32_32x32x16_bf16).
//
// Operands are copied from global memory to LDS by global_load_lds_dwordx4 (16 bytes per
// lane, no register staging) in one of two LDS layouts, chosen to match global memory:
//   KC: [row][k]  (k contiguous)   -- fragments read with ds_read_b128;
//   MC: [k][row]  (rows contiguous) -- fragments read with two ds_read_b64_tr_b16, which
//       hand lane i of each 16-lane group column (i mod 4) of the rows addressed by lanes
//       {i/4, 4+i/4, 8+i/4, 12+i/4}; addressing rows k.. and columns n.. accordingly
//       yields the 8-element k-run of column n that the matrix core expects.
// 16-byte slots within an LDS row are XOR-swizzled by a function of the row so that the
// fragment reads of neighbouring rows fall in different banks.
// NS LDS stages form a ring; the copy of k-tile t+NS-1 runs while tile t is consumed.
// Out-of-range rows or k read from a 16-byte zero page, so ragged tiles need no masking.
#pragma once

#include "pctc_device.h"

namespace pctc {
namespace bf {

enum class LL { KC, MC };

__device__ __attribute__((aligned(16))) static const uint32_t kZeroPage[4] = {0u, 0u, 0u, 0u};

struct GOp {
  const uint16_t* base;
  int64_t pitch;        // elements between consecutive rows (KC) or k-lines (MC)
  int rows;             // valid rows
  int kmax;             // valid k
  const int* rowidx;    // KC only: optional row gather table
};

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((ext_vector_type(4))) short s16x4;

__device__ __forceinline__ void lds_copy16(const void* g, lds_void* l) {
  __builtin_amdgcn_global_load_lds(g, l, 16, 0, 0);
}

// vmcnt <= n (n < 64), other counters unconstrained.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

template <int BK>
struct KC {
  static constexpr int kSlots = BK / 8;          // 16-byte slots per row
  static constexpr int kRowBytes = BK * 2;
  static constexpr int kRowsPerCopy = 64 / kSlots;
  __device__ static __forceinline__ int swz(int r) {
    if constexpr (BK == 64) return r & 7;
    else return (r >> 2) & 3;
  }
};

template <int R>
struct MC {
  static constexpr int kSlots = R / 8;
  static constexpr int kRowBytes = R * 2;
  static constexpr int kRowsPerCopy = 64 / kSlots;
  __device__ static __forceinline__ int swz(int kr) { return ((kr & 7) << 1) & (kSlots - 1); }
};

// Copies one operand tile (NR rows x BK k) into LDS as kCopies 1 KB copies; wave w of
// NW issues copies w, w+NW, ...  Per-copy source offsets are fixed for the whole k loop
// and are computed once (init); issue() adds the k-tile offset.
template <LL L, int NR, int BK, int NW>
struct TileCopy {
  static constexpr int kBytes = NR * BK * 2;
  static constexpr int kCopies = kBytes / 1024;
  static constexpr int kPerWave = kCopies / NW;
  static_assert(kBytes % 1024 == 0 && kCopies % NW == 0, "tile must be whole 1 KB copies per wave");
  const uint16_t* src[kPerWave];
  int lim[kPerWave];  // KC: k-offset of this lane's slot; MC: k-line of this lane
  bool ok[kPerWave];  // row in range

  __device__ __forceinline__ void init(const GOp& op, int row0, int w, int lane) {
#pragma unroll
    for (int i = 0; i < kPerWave; ++i) {
      const int c = w + NW * i;
      if constexpr (L == LL::KC) {
        using G = KC<BK>;
        const int r = c * G::kRowsPerCopy + lane / G::kSlots;
        const int lc = (lane % G::kSlots) ^ G::swz(r);
        const int row = row0 + r;
        ok[i] = row < op.rows;
        int64_t grow = row;
        if (op.rowidx) grow = ok[i] ? op.rowidx[row] : 0;
        src[i] = op.base + grow * op.pitch + lc * 8;
        lim[i] = lc * 8;
      } else {
        using G = MC<NR>;
        const int kr = c * G::kRowsPerCopy + lane / G::kSlots;
        const int lc = (lane % G::kSlots) ^ G::swz(kr);
        const int row = row0 + lc * 8;
        ok[i] = row < op.rows;
        src[i] = op.base + static_cast<int64_t>(kr) * op.pitch + row;
        lim[i] = kr;
      }
    }
  }

  // Same as init for a tile whose first row is row0 (no row gather).
  __device__ __forceinline__ void retarget(const GOp& op, int row0, int w, int lane) {
#pragma unroll
    for (int i = 0; i < kPerWave; ++i) {
      const int c = w + NW * i;
      if constexpr (L == LL::KC) {
        using G = KC<BK>;
        const int r = c * G::kRowsPerCopy + lane / G::kSlots;
        const int row = row0 + r;
        ok[i] = row < op.rows;
        src[i] = op.base + static_cast<int64_t>(row) * op.pitch + lim[i];
      } else {
        using G = MC<NR>;
        const int lc = (lane % G::kSlots) ^ G::swz(lim[i]);
        const int row = row0 + lc * 8;
        ok[i] = row < op.rows;
        src[i] = op.base + static_cast<int64_t>(lim[i]) * op.pitch + row;
      }
    }
  }

  __device__ __forceinline__ void issue(const GOp& op, int k0, char* lds, int w) const {
#pragma unroll
    for (int i = 0; i < kPerWave; ++i) {
      const int c = w + NW * i;
      const bool valid = ok[i] && (k0 + lim[i] < op.kmax);
      const int64_t koff = (L == LL::KC) ? static_cast<int64_t>(k0) : static_cast<int64_t>(k0) * op.pitch;
      const void* g = valid ? static_cast<const void*>(src[i] + koff) : static_cast<const void*>(kZeroPage);
      lds_copy16(g, (lds_void*)(lds + c * 1024));
    }
  }
};

// 8-element bf16 fragment of row (or column) `rr` for k in [kk + 8h, kk + 8h + 8).
template <LL L, int NR, int BK>
__device__ __forceinline__ bf16x8 frag(const char* lds, int rr_base, int kk, int lane) {
  if constexpr (L == LL::KC) {
    using G = KC<BK>;
    const int r = rr_base + (lane & 31);
    const int c = (kk >> 3) + (lane >> 5);
    const int off = r * G::kRowBytes + ((c ^ G::swz(r)) << 4);
    return *reinterpret_cast<const bf16x8*>(lds + off);
  } else {
    using G = MC<NR>;
    const int h = lane >> 5, g2 = (lane >> 4) & 1, j = lane & 15;
    const int n = rr_base + 16 * g2 + 4 * (j & 3);
    const int c = n >> 3, half = (n >> 2) & 1;
    s16x4 v[2];
#pragma unroll
    for (int rd = 0; rd < 2; ++rd) {
      const int kr = kk + 8 * h + 4 * rd + (j >> 2);
      const int off = kr * G::kRowBytes + ((c ^ G::swz(kr)) << 4) + (half << 3);
      v[rd] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(lds + off));
    }
    bf16x8 out;
    __builtin_memcpy(&out, v, 16);
    return out;
  }
}

// NS-stage ring with one barrier per k-tile.  Iteration t: wait until this wave's copies
// of tile t have landed (later tiles may still be in flight), barrier (tile t visible to
// every wave; every wave is done reading tile t-1's stage), issue the copy of tile
// t+NS-1 into that freed stage, then consume tile t.  The k loop is unrolled by NS so
// that each stage is a distinct LDS object: the compiler can see that reading one stage
// does not depend on copies in flight into the others.
// Waves form a WR x WC grid; each owns (BR/WR) x (BC/WC) = FR x FC blocks of 32x32.
template <int BR, int BC, int BK, LL LA, LL LB, int NS, int WR = 2, int WC = 2>
struct Gemm {
  static constexpr int kNS = NS;
  static constexpr int kBR = BR, kBC = BC;
  static constexpr int NW = WR * WC;
  static constexpr int kThreads = 64 * NW;
  static constexpr int FR = BR / WR / 32, FC = BC / WC / 32;
  static constexpr int kABytes = BR * BK * 2;
  static constexpr int kBBytes = BC * BK * 2;
  static constexpr int kStageBytes = kABytes + kBBytes;
  using CA = TileCopy<LA, BR, BK, NW>;
  using CB = TileCopy<LB, BC, BK, NW>;
  static constexpr int kCopiesPerWave = CA::kPerWave + CB::kPerWave;
  static_assert(NS >= 2 && NS <= 4, "stages");
  static_assert(kCopiesPerWave * (NS - 1) < 64, "vmcnt range");

  // Row (within the tile) of accumulator register r of block i, and column of block j.
  __device__ static __forceinline__ int row_of(int wave, int lane, int i, int r) {
    return (wave / WC) * (BR / WR) + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
  }
  __device__ static __forceinline__ int col_of(int wave, int lane, int j) {
    return (wave % WC) * (BC / WC) + 32 * j + (lane & 31);
  }

  __device__ static __forceinline__ void compute(const char* stage, int wave, int lane, f32x16 (&acc)[FR][FC]) {
    const char* la = stage;
    const char* lb = stage + kABytes;
    const int wr0 = (wave / WC) * (BR / WR);
    const int wc0 = (wave % WC) * (BC / WC);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8 a[FR], b[FC];
#pragma unroll
      for (int i = 0; i < FR; ++i) a[i] = frag<LA, BR, BK>(la, wr0 + 32 * i, kk, lane);
#pragma unroll
      for (int j = 0; j < FC; ++j) b[j] = frag<LB, BC, BK>(lb, wc0 + 32 * j, kk, lane);
#pragma unroll
      for (int i = 0; i < FR; ++i)
#pragma unroll
        for (int j = 0; j < FC; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  }

  template <int S>
  __device__ static __forceinline__ void step(const GOp& A, const GOp& B, const CA& ca, const CB& cb, int kbeg, int kt,
                                              int nk, char* const (&st)[NS], int wave, int lane,
                                              f32x16 (&acc)[FR][FC]) {
    // copies issued after tile kt so far: tiles kt+1 .. min(kt+NS-2, nk-1)
    const int after = min(NS - 2, nk - 1 - kt);
    if constexpr (NS >= 4) {
      if (after >= 2) wait_vmcnt<2 * kCopiesPerWave>();
      else if (after == 1) wait_vmcnt<kCopiesPerWave>();
      else wait_vmcnt<0>();
    } else if constexpr (NS == 3) {
      if (after >= 1) wait_vmcnt<kCopiesPerWave>();
      else wait_vmcnt<0>();
    } else {
      wait_vmcnt<0>();
    }
    __builtin_amdgcn_s_barrier();
    const int nt = kt + NS - 1;
    if (nt < nk) {
      constexpr int SN = (S + NS - 1) % NS;
      ca.issue(A, kbeg + nt * BK, st[SN], wave);
      cb.issue(B, kbeg + nt * BK, st[SN] + kABytes, wave);
    }
    compute(st[S], wave, lane, acc);
  }

  // A sequence of ntiles output tiles sharing the B rows (col0) and the k range [0, K):
  // tile i uses A rows from row0 + i * BR.  The copy pipeline runs straight through the
  // tile boundaries; epi(i, acc) is called after tile i's last product (while the copy of
  // the next tile's first k-tile is in flight) and must not touch the LDS stages.
  template <class Epi>
  __device__ static __forceinline__ void run_tiles(const GOp& A, const GOp& B, int row0, int col0, int ntiles, int K,
                                                   char* const (&st)[NS], f32x16 (&acc)[FR][FC], Epi&& epi) {
    static_assert(NS == 2, "flattened sequence uses two stages");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nk = (K + BK - 1) / BK;
    const int nsteps = ntiles * nk;
    CA ca;
    CB cb;
    ca.init(A, row0, wave, lane);
    cb.init(B, col0, wave, lane);
#pragma unroll
    for (int i = 0; i < FR; ++i)
#pragma unroll
      for (int j = 0; j < FC; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    __builtin_amdgcn_s_barrier();
    if (nsteps <= 0) return;
    ca.issue(A, 0, st[0], wave);
    cb.issue(B, 0, st[0] + kABytes, wave);
    wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    auto half = [&](int sidx, char* cur, char* nxt) {
      const int tile = sidx / nk, kt = sidx - tile * nk;
      if (sidx + 1 < nsteps) {
        const int kn = (kt + 1 == nk) ? 0 : kt + 1;
        if (kn == 0) ca.retarget(A, row0 + (tile + 1) * BR, wave, lane);
        ca.issue(A, kn * BK, nxt, wave);
        cb.issue(B, kn * BK, nxt + kABytes, wave);
      }
      compute(cur, wave, lane, acc);
      if (kt == nk - 1) {
        epi(tile, acc);
#pragma unroll
        for (int i = 0; i < FR; ++i)
#pragma unroll
          for (int j = 0; j < FC; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
      }
      wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();
    };
    for (int sidx = 0; sidx < nsteps; sidx += 2) {
      half(sidx, st[0], st[1]);
      if (sidx + 1 < nsteps) half(sidx + 1, st[1], st[0]);
    }
  }

  // Accumulates k in [kbeg, kend) (kbeg a multiple of BK) into acc (zeroed here).
  // All kThreads threads must call; contains barriers.  st[s]: kStageBytes each.
  __device__ static __forceinline__ void run(const GOp& A, const GOp& B, int row0, int col0, int kbeg, int kend,
                                             char* const (&st)[NS], f32x16 (&acc)[FR][FC]) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
#pragma unroll
    for (int i = 0; i < FR; ++i)
#pragma unroll
      for (int j = 0; j < FC; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    const int nk = (kend - kbeg + BK - 1) / BK;
    CA ca;
    CB cb;
    ca.init(A, row0, wave, lane);
    cb.init(B, col0, wave, lane);
    __builtin_amdgcn_s_barrier();  // previous users of the stages are done
#pragma unroll
    for (int s = 0; s < NS - 1; ++s) {
      if (s < nk) {
        ca.issue(A, kbeg + s * BK, st[s], wave);
        cb.issue(B, kbeg + s * BK, st[s] + kABytes, wave);
      }
    }
    for (int kt = 0; kt < nk; kt += NS) {
      step<0>(A, B, ca, cb, kbeg, kt, nk, st, wave, lane, acc);
      if (kt + 1 < nk) step<1>(A, B, ca, cb, kbeg, kt + 1, nk, st, wave, lane, acc);
      if constexpr (NS >= 3)
        if (kt + 2 < nk) step<2 % NS>(A, B, ca, cb, kbeg, kt + 2, nk, st, wave, lane, acc);
      if constexpr (NS >= 4)
        if (kt + 3 < nk) step<3 % NS>(A, B, ca, cb, kbeg, kt + 3, nk, st, wave, lane, acc);
    }
  }
};

// ---------------------------------------------------------------------------------------
// Variant with one operand loaded straight into registers.
//
// The LDS copy path has limited throughput, so one operand (the "direct" one, which must
// be K-contiguous in global memory) bypasses LDS: each lane loads its own 16-byte MFMA
// fragments with ordinary vector loads, one k-tile ahead into a register double buffer.
// The other operand goes through a two-stage LDS ring as above.  Within a k-tile of BK,
// lane half h owns k in [h BK/2, (h+1) BK/2) and step s uses the s-th 8-run of it, so a
// lane's direct loads for one k-tile are contiguous.
// ---------------------------------------------------------------------------------------

__device__ __forceinline__ int kidx_of(int BKh, int s, int lane) { return BKh * (lane >> 5) + 8 * s; }

template <LL L, int NR, int BK>
__device__ __forceinline__ bf16x8 frag_k(const char* lds, int rr_base, int kidx, int lane) {
  if constexpr (L == LL::KC) {
    using G = KC<BK>;
    const int r = rr_base + (lane & 31);
    const int c = kidx >> 3;
    const int off = r * G::kRowBytes + ((c ^ G::swz(r)) << 4);
    return *reinterpret_cast<const bf16x8*>(lds + off);
  } else {
    using G = MC<NR>;
    const int g2 = (lane >> 4) & 1, j = lane & 15;
    const int n = rr_base + 16 * g2 + 4 * (j & 3);
    const int c = n >> 3, half = (n >> 2) & 1;
    s16x4 v[2];
#pragma unroll
    for (int rd = 0; rd < 2; ++rd) {
      const int kr = kidx + 4 * rd + (j >> 2);
      const int off = kr * G::kRowBytes + ((c ^ G::swz(kr)) << 4) + (half << 3);
      v[rd] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(lds + off));
    }
    bf16x8 out;
    __builtin_memcpy(&out, v, 16);
    return out;
  }
}

// Fragments of NB 32-row blocks of a K-contiguous operand for one k-tile, loaded by this lane.
template <int NB, int BK>
struct Direct {
  static constexpr int KS = BK / 16;
  const uint16_t* src[NB];
  bool ok[NB];
  __device__ __forceinline__ void init(const GOp& op, int rowbase, int lane) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int row = rowbase + 32 * b + (lane & 31);
      ok[b] = row < op.rows;
      int64_t grow = row;
      if (op.rowidx) grow = ok[b] ? op.rowidx[row] : 0;
      src[b] = op.base + grow * op.pitch + (BK / 2) * (lane >> 5);
    }
  }
  __device__ __forceinline__ void load(const GOp& op, int k0, int lane, bf16x8 (&f)[NB][KS]) const {
    const int kb = k0 + (BK / 2) * (lane >> 5);
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const bool valid = ok[b] && (kb + 8 * s < op.kmax);
        const bf16x8* p = valid ? reinterpret_cast<const bf16x8*>(src[b] + k0 + 8 * s)
                                : reinterpret_cast<const bf16x8*>(kZeroPage);
        f[b][s] = *p;
      }
  }
};

// DIRECT = 1: A direct, B through LDS.  DIRECT = 2: B direct, A through LDS.
template <int BR, int BC, int BK, LL LL_LDS, int DIRECT, int WR = 2, int WC = 2>
struct GemmD {
  static constexpr int NW = WR * WC;
  static constexpr int kThreads = 64 * NW;
  static constexpr int kBR = BR, kBC = BC;
  static constexpr int FR = BR / WR / 32, FC = BC / WC / 32;
  static constexpr int KS = BK / 16;
  static constexpr int kLdsRows = (DIRECT == 1) ? BC : BR;
  static constexpr int kStageBytes = kLdsRows * BK * 2;
  static constexpr int ND = (DIRECT == 1) ? FR : FC;  // direct blocks per wave
  static constexpr int NL = (DIRECT == 1) ? FC : FR;  // LDS blocks per wave
  using CL = TileCopy<LL_LDS, kLdsRows, BK, NW>;
  using DR = Direct<ND, BK>;

  __device__ static __forceinline__ int row_of(int wave, int lane, int i, int r) {
    return (wave / WC) * (BR / WR) + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
  }
  __device__ static __forceinline__ int col_of(int wave, int lane, int j) {
    return (wave % WC) * (BC / WC) + 32 * j + (lane & 31);
  }

  __device__ static __forceinline__ void compute(const char* stage, const bf16x8 (&d)[ND][KS], int wave, int lane,
                                                 f32x16 (&acc)[FR][FC]) {
    const int wr0 = (wave / WC) * (BR / WR);
    const int wc0 = (wave % WC) * (BC / WC);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int kidx = kidx_of(BK / 2, s, lane);
      bf16x8 l[NL];
#pragma unroll
      for (int t = 0; t < NL; ++t)
        l[t] = frag_k<LL_LDS, kLdsRows, BK>(stage, (DIRECT == 1 ? wc0 : wr0) + 32 * t, kidx, lane);
#pragma unroll
      for (int i = 0; i < FR; ++i)
#pragma unroll
        for (int j = 0; j < FC; ++j) {
          if constexpr (DIRECT == 1)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(d[i][s], l[j], acc[i][j], 0, 0, 0);
          else
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(l[i], d[j][s], acc[i][j], 0, 0, 0);
        }
    }
  }

  // Accumulates k in [kbeg, kend) (kbeg a multiple of BK) into acc (zeroed here).
  // A and B as in Gemm; the direct operand must be KC.  All kThreads threads must call.
  __device__ static __forceinline__ void run(const GOp& A, const GOp& B, int row0, int col0, int kbeg, int kend,
                                             char* st0, char* st1, f32x16 (&acc)[FR][FC]) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
#pragma unroll
    for (int i = 0; i < FR; ++i)
#pragma unroll
      for (int j = 0; j < FC; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    const GOp& OL = (DIRECT == 1) ? B : A;
    const GOp& OD = (DIRECT == 1) ? A : B;
    const int lbase = (DIRECT == 1) ? col0 : row0;
    const int dbase = (DIRECT == 1) ? row0 + (wave / WC) * (BR / WR) : col0 + (wave % WC) * (BC / WC);
    const int nk = (kend - kbeg + BK - 1) / BK;
    CL cl;
    DR dr;
    cl.init(OL, lbase, wave, lane);
    dr.init(OD, dbase, lane);
    bf16x8 d0[ND][KS], d1[ND][KS];
    __builtin_amdgcn_s_barrier();  // previous users of st0/st1 are done
    if (nk <= 0) return;
    cl.issue(OL, kbeg, st0, wave);
    dr.load(OD, kbeg, lane, d0);
    wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    const int npairs = nk >> 1;
    for (int p = 0; p < npairs; ++p) {
      const int kt = 2 * p;
      cl.issue(OL, kbeg + (kt + 1) * BK, st1, wave);
      dr.load(OD, kbeg + (kt + 1) * BK, lane, d1);
      compute(st0, d0, wave, lane, acc);
      wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();
      if (kt + 2 < nk) {
        cl.issue(OL, kbeg + (kt + 2) * BK, st0, wave);
        dr.load(OD, kbeg + (kt + 2) * BK, lane, d0);
      }
      compute(st1, d1, wave, lane, acc);
      wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();
    }
    if (nk & 1) compute(st0, d0, wave, lane, acc);
  }
};

}  // namespace bf
}  // namespace pctc
