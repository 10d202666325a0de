// bf16 matrix-core tile engine for gfx950 with direct global->LDS staging.
//
// C[i][j] = sum_k A[i][k] B[j][k] over one BR x BC tile (WR x WC wavefronts, 4 or 8; each owns
// (BR/WR) x (BC/WC) = FR x FC blocks of 32x32 accumulated by v_mfma_f32_32x32x16_bf16).
//
// Operands are copied from global memory to LDS by buffer_load_dwordx4 ... lds (16 bytes per
// lane, no register staging) in one of two LDS layouts, chosen to match global memory:
//   KC: [row][k]  (k contiguous)   -- fragments read with ds_read_b128;
//   MC: [k][row]  (rows contiguous) -- fragments read with two ds_read_b64_tr_b16, which
//       hand lane i of each 16-lane group column (i mod 4) of the rows addressed by lanes
//       {i/4, 4+i/4, 8+i/4, 12+i/4}; addressing rows k.. and columns n.. accordingly
//       yields the 8-element k-run of column n that the matrix core expects.
// 16-byte slots within an LDS row are XOR-swizzled by a function of the row so that the
// fragment reads of neighbouring rows fall in different banks.
// NS LDS stages form a ring: while k-tile t is consumed, the copies of tiles t+1..t+NS-1
// are in flight, and the copy of t+NS is issued as soon as every wave has read tile t.
// Fragments are double-buffered in registers across k-steps, and every k-step issues its
// matrix products interleaved one by one with the next step's LDS reads (and copies), so
// the matrix pipe is fed while the reads are in flight.
// Out-of-range rows and k read zeros, so ragged tiles need no masking: each k-tile's copies
// go through a buffer resource whose base and size (scalar registers) cover exactly the
// tile's valid part, and the hardware returns zero for every lane whose offset falls past
// the size (lanes of invalid columns or k carry bit 31 in their fixed offset).  A copy then
// costs no vector arithmetic.  Row-gathered operands (GOp::rowidx) keep per-lane addresses
// with a 16-byte zero page.  The k loop runs a multiple of NS tiles (the extra tiles are
// zeros).
// Schedules: Gemm::run / run_seq / run_seq_aligned interleave products and reads in every
// wave (one barrier per k-tile); Gemm::run_pp (8 waves) alternates two groups of four waves
// between a memory phase and a products-only phase.  GemmA64 (ping-pong) and GemmMidA64 (tile
// runs with epilogues) copy a k-contiguous operand 64 deep, so that each of its row pieces is
// a whole 128-byte line: a 64-byte piece costs the cache about as much as a whole line.
#pragma once

#include "pctc_device.h"

namespace pctc {
namespace bf {

enum class LL { KC, MC };

__device__ __attribute__((aligned(16))) static const uint32_t kZeroPage[4] = {0u, 0u, 0u, 0u};

struct GOp {
  const uint16_t* base;
  int64_t pitch;        // elements between consecutive rows (KC) or k-lines (MC); MC: rows <= pitch
  int rows;             // valid rows
  int kmax;             // valid k (KC: kmax <= pitch)
  const int* rowidx;    // KC only: optional row gather table (needs a Gemm with BUF false)
};

// Word 3 of a raw buffer resource on gfx9-family parts: 32-bit data format, no swizzle.
constexpr int kBufWord3 = 0x00020000;
constexpr uint32_t kOob = 0x80000000u;  // an offset past any size used here

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
  // A ds_read_b128 phase serves 16 lanes (16 rows) from 64 banks of 4 bytes: rows of 128 bytes
  // (BK = 64) put even and odd rows in different halves of the banks, so the slot is XORed with
  // (r >> 1) mod 8 (eight different slots among the even rows of a phase, eight among the odd);
  // rows of 64 bytes (BK = 32) fill a 256-byte bank line four at a time.
  __device__ static __forceinline__ int swz(int r) {
    if constexpr (BK == 64) return (r >> 1) & 7;
    else return (r >> 2) & 3;
  }
};

template <int R>
struct MC {
  static constexpr int kSlots = R / 8;
  static constexpr int kRowBytes = R * 2;
  static constexpr int kRowsPerCopy = 64 / kSlots;
  // A transpose read takes, per half-wavefront, 4 consecutive k-lines x 4 consecutive slots:
  // k-line kr moves its slots by (kr mod 4) groups of 4, so the 16 reads land in 16
  // different 16-byte bank groups.
  __device__ static __forceinline__ int swz(int kr) { return ((kr & 3) << 2) & (kSlots - 1); }
};

// Copies one operand tile (NR rows x BK k) into LDS as kCopies 1 KB copies; wave w of
// NW issues copies w, w+NW, ...  Per-copy source offsets are fixed for the whole k loop
// and are computed once (init); issue() adds the k-tile offset.  BUF: through buffer
// resources (below); otherwise flat addresses with the zero page (row gathers).
template <LL L, int NR, int BK, int NW, bool BUF>
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

  // Copies k-tile [k0, k0 + BK); k at or past klim reads zeros.
  __device__ __forceinline__ void issue(const GOp& op, int k0, int klim, char* lds, int w) const {
#pragma unroll
    for (int i = 0; i < kPerWave; ++i) {
      const int c = w + NW * i;
      const bool valid = ok[i] && (k0 + lim[i] < klim);
      const int64_t koff = (L == LL::KC) ? static_cast<int64_t>(k0) : static_cast<int64_t>(k0) * op.pitch;
      const void* g = valid ? static_cast<const void*>(src[i] + koff) : static_cast<const void*>(kZeroPage);
      lds_copy16(g, (lds_void*)(lds + c * 1024));
    }
  }
};

// Buffer-resource copies.  Byte offsets of a lane's 16 bytes, relative to the k-tile base
// (KC: row row0, element k0; MC: k-line k0, element row0):
//   KC: r pitch 2 + 16 slot   valid while r < rows - row0 (the size stops there) and
//                              k0 + 8 slot < klim (only the one partial k-tile can break
//                              this: there, lanes past the limit add bit 31; a lane's slot
//                              is the same in all its copies, so one flag covers them);
//   MC: kr pitch 2 + 16 slot  valid while k0 + kr < klim (the size stops at that k-line)
//                              and row0 + 8 slot < rows (otherwise bit 31 is set).
// With 16-byte reads that either lie wholly below the size or start at or past it.
template <LL L, int NR, int BK, int NW>
struct TileCopy<L, NR, BK, NW, true> {
  static constexpr int kBytes = NR * BK * 2;
  static constexpr int kCopies = kBytes / 1024;
  static constexpr int kPerWave = kCopies / NW;
  static_assert(kBytes % 1024 == 0 && kCopies % NW == 0, "tile must be whole 1 KB copies per wave");
  const uint16_t* tbase;  // KC: op.base + row0 pitch; MC: op.base + row0
  int rows_left;          // KC: valid rows of the tile (0 .. NR); MC: row0
  int kpart;              // KC: k0 of the partial k-tile (none: -1)
  uint32_t poob;          // KC: bit 31 if this lane's slot is past the partial k-tile's limit
  uint32_t off[kPerWave];

  __device__ __forceinline__ void init(const GOp& op, int row0, int w, int lane, int kbeg, int klim) {
    const int rem = (klim > kbeg) ? (klim - kbeg) % BK : 0;
    kpart = rem ? klim - rem : -1;
#pragma unroll
    for (int i = 0; i < kPerWave; ++i) {
      const int c = w + NW * i;
      if constexpr (L == LL::KC) {
        using G = KC<BK>;
        const int r = c * G::kRowsPerCopy + lane / G::kSlots;
        const int lc = (lane % G::kSlots) ^ G::swz(r);
        off[i] = static_cast<uint32_t>(r * op.pitch * 2 + lc * 16);
        poob = (lc * 8 < rem) ? 0u : kOob;  // the same for every i
      } else {
        using G = MC<NR>;
        const int kr = c * G::kRowsPerCopy + lane / G::kSlots;
        const int lc = (lane % G::kSlots) ^ G::swz(kr);
        off[i] = static_cast<uint32_t>(kr * op.pitch * 2 + lc * 16) | ((row0 + lc * 8 < op.rows) ? 0u : kOob);
      }
    }
    if constexpr (L == LL::MC) rows_left = row0;  // the offsets above are this tile's
    retarget(op, row0, w, lane);
  }

  // The tile whose first row is row0 (same k range).
  __device__ __forceinline__ void retarget(const GOp& op, int row0, int w, int lane) {
    if constexpr (L == LL::KC) {
      tbase = op.base + static_cast<int64_t>(row0) * op.pitch;
      rows_left = min(max(op.rows - row0, 0), NR);
    } else {
      tbase = op.base + row0;
      if (row0 != rows_left) {  // column validity moves with the tile
#pragma unroll
        for (int i = 0; i < kPerWave; ++i) {
          const int c = w + NW * i;
          using G = MC<NR>;
          const int kr = c * G::kRowsPerCopy + lane / G::kSlots;
          const int lc = (lane % G::kSlots) ^ G::swz(kr);
          off[i] = static_cast<uint32_t>(kr * op.pitch * 2 + lc * 16) | ((row0 + lc * 8 < op.rows) ? 0u : kOob);
        }
      }
      rows_left = row0;
    }
  }

  __device__ __forceinline__ void issue(const GOp& op, int k0, int klim, char* lds, int w) const {
#if defined(__HIP_DEVICE_COMPILE__)  // the buffer-resource type exists on the device side only
    // 32-bit sizes (NR or BK pitch-long rows or k-lines) and a base made explicitly uniform, so
    // that the resource sits in scalar registers (a per-lane resource would be looped over)
    const int p2 = static_cast<int>(op.pitch) * 2;
    int size;
    const uint16_t* b;
    if constexpr (L == LL::KC) {
      b = tbase + k0;
      size = (k0 < klim) ? rows_left * p2 - k0 * 2 : 0;
    } else {
      b = tbase + static_cast<int64_t>(k0) * op.pitch;
      // (klim - k0 <= 0 leaves size <= 0: no k-line of this tile is valid)
      size = min(klim - k0, BK) * p2 - rows_left * 2;
    }
    size = __builtin_amdgcn_readfirstlane(max(size, 0));
    const uint64_t ba = reinterpret_cast<uint64_t>(b);
    const uint64_t bu = (static_cast<uint64_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(ba >> 32))) << 32) |
                        static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(ba)));
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(bu),
                                                                       static_cast<short>(0), size, kBufWord3);
    uint32_t adj = 0u;
    if constexpr (L == LL::KC) {
      adj = (k0 == kpart) ? poob : 0u;
      asm volatile("" : "+v"(adj));  // one register per issue, not a hoisted second offset set
    }
#pragma unroll
    for (int i = 0; i < kPerWave; ++i) {
      const int c = w + NW * i;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(lds + c * 1024), 16, off[i] | adj, 0, 0, 0);
    }
#endif
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

// Tile engine.  Waves form a WR x WC grid; each owns (BR/WR) x (BC/WC) = FR x FC blocks of
// 32x32.  BK must be a multiple of 32 (an even number of 16-deep k-steps per tile).  PRE: in a
// tile's last k-step, half of the products are issued before the barrier (they need only
// registers), so the matrix pipe has work while the wave waits there; this pays where one
// workgroup fills the CU (no other workgroup's products to fill the wait).
template <int BR, int BC, int BK, LL LA, LL LB, int NS, int WR = 2, int WC = 2, bool PRE = false, bool BUF = true>
struct Gemm {
  static constexpr int kNS = NS;
  static constexpr int kBR = BR, kBC = BC;
  static constexpr int NW = WR * WC;
  static constexpr int kThreads = 64 * NW;
  static constexpr int FR = BR / WR / 32, FC = BC / WC / 32;
  static constexpr int KK = BK / 16;
  static constexpr int kABytes = BR * BK * 2;
  static constexpr int kBBytes = BC * BK * 2;
  static constexpr int kStageBytes = kABytes + kBBytes;
  // bytes of each stage array a kernel declares for this engine (engines that declare their
  // own stages set it to a stub)
  static constexpr int kKernelStageBytes = kStageBytes;
  using CA = TileCopy<LA, BR, BK, NW, BUF>;
  using CB = TileCopy<LB, BC, BK, NW, BUF>;
  static constexpr int CPW = CA::kPerWave + CB::kPerWave;  // copies per wave per k-tile
  static_assert(NS >= 2 && NS <= 4, "stages");
  static_assert(KK % 2 == 0, "BK must be a multiple of 32");
  static_assert(CPW * NS < 64, "vmcnt range");
  // LDS reads per fragment set (the transpose read takes two per fragment)
  static constexpr int ND = FR * (LA == LL::MC ? 2 : 1) + FC * (LB == LL::MC ? 2 : 1);
  static constexpr int NM = FR * FC;

  struct Frags {
    bf16x8 a[FR], b[FC];
  };

  // Row (within the tile) of accumulator register r of block i, and column of block j.
  __device__ static __forceinline__ int row_of(int wave, int lane, int i, int r) {
    return (wave / WC) * (BR / WR) + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
  }
  __device__ static __forceinline__ int col_of(int wave, int lane, int j) {
    return (wave % WC) * (BC / WC) + 32 * j + (lane & 31);
  }

  __device__ static __forceinline__ void zero(f32x16 (&acc)[FR][FC]) {
#pragma unroll
    for (int i = 0; i < FR; ++i)
#pragma unroll
      for (int j = 0; j < FC; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  }

  __device__ static __forceinline__ void load(const char* stage, int kk, int wave, int lane, Frags& f) {
    const int wr0 = (wave / WC) * (BR / WR), wc0 = (wave % WC) * (BC / WC);
#pragma unroll
    for (int i = 0; i < FR; ++i) f.a[i] = frag<LA, BR, BK>(stage, wr0 + 32 * i, kk * 16, lane);
#pragma unroll
    for (int j = 0; j < FC; ++j) f.b[j] = frag<LB, BC, BK>(stage + kABytes, wc0 + 32 * j, kk * 16, lane);
  }

  // products q in [B, E) of the FR x FC blocks (q = i FC + j)
  template <int B, int E>
  __device__ static __forceinline__ void mma_range(const Frags& f, f32x16 (&acc)[FR][FC]) {
#pragma unroll
    for (int q = B; q < E; ++q)
      acc[q / FC][q % FC] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[q / FC], f.b[q % FC], acc[q / FC][q % FC], 0, 0, 0);
  }

  __device__ static __forceinline__ void mma(const Frags& f, f32x16 (&acc)[FR][FC]) {
#pragma unroll
    for (int i = 0; i < FR; ++i)
#pragma unroll
      for (int j = 0; j < FC; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
  }

  // Instruction order of one k-step: each matrix product is followed by its share of the
  // ND reads of the next step and, in a tile's last step, of the NV copies.
  template <int NV, int NMM = NM>
  __device__ static __forceinline__ void interleave() {
#pragma unroll
    for (int q = 0; q < NMM; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one matrix product
      if (q < NV) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // one global load
      const int d = (q + 1) * ND / NMM - q * ND / NMM;
      if (d == 1) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS reads
      else if (d == 2) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      else if (d == 3) __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
      else if (d >= 4) __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  }

  // One k-tile held in stage S; the fragments of its first k-step are in f0.  In the last
  // k-step: wait for this wave's copies of the next tile, barrier (the next tile is
  // visible and every wave is done reading stage S), then `issue` refills stage S and
  // the next tile's first fragments are read into f0 (stage S+1).
  //
  // XTRA > 0 (run_seq_aligned): at least XTRA vector memory instructions (an epilogue's
  // stores) were issued after the copies this wait is for, so the wait leaves that many more
  // outstanding (the counter completes in issue order) and the stores drain under the
  // products.
  template <int S, int XTRA = 0, class Issue>
  __device__ static __forceinline__ void ktile(char* const (&st)[NS], int wave, int lane, f32x16 (&acc)[FR][FC],
                                               Frags& f0, Frags& f1, Issue&& issue) {
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      Frags& cur = (kk & 1) ? f1 : f0;
      Frags& nxt = (kk & 1) ? f0 : f1;
      if (kk + 1 < KK) {
        load(st[S], kk + 1, wave, lane, nxt);
        mma(cur, acc);
        interleave<0>();
      } else {
        constexpr int NH = PRE ? NM / 2 : 0;
        if constexpr (PRE) mma_range<0, NH>(cur, acc);
        static_assert((NS - 2) * CPW + XTRA < 64, "vmcnt range");
        wait_vmcnt<(NS - 2) * CPW + XTRA>();
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's reads of stage S are done
        __builtin_amdgcn_s_barrier();
        issue(st[S]);
        load(st[(S + 1) % NS], 0, wave, lane, nxt);
        mma_range<NH, NM>(cur, acc);
        interleave<CPW, NM - NH>();
      }
    }
  }

  // Accumulates k in [kbeg, kend) (kbeg a multiple of BK) into acc (zeroed here unless
  // ZERO is false, when acc holds starting values).  All kThreads threads must call;
  // contains barriers.  st[s]: kStageBytes each.  On return every copy has landed and
  // every wave is past its last LDS read.
  template <bool ZERO = true>
  __device__ static __forceinline__ void run(const GOp& A, const GOp& B, int row0, int col0, int kbeg, int kend,
                                             char* const (&st)[NS], f32x16 (&acc)[FR][FC]) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: copy targets in scalar registers
    if constexpr (ZERO) zero(acc);
    const int nk = (kend - kbeg + BK - 1) / BK;
    if (nk <= 0) return;
    const int klimA = min(A.kmax, kend), klimB = min(B.kmax, kend);
    CA ca;
    CB cb;
    if constexpr (BUF) {
      ca.init(A, row0, wave, lane, kbeg, klimA);
      cb.init(B, col0, wave, lane, kbeg, klimB);
    } else {
      ca.init(A, row0, wave, lane);
      cb.init(B, col0, wave, lane);
    }
    __builtin_amdgcn_s_barrier();  // previous users of the stages are done
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      ca.issue(A, kbeg + s * BK, klimA, st[s], wave);
      cb.issue(B, kbeg + s * BK, klimB, st[s] + kABytes, wave);
    }
    wait_vmcnt<(NS - 1) * CPW>();
    __builtin_amdgcn_s_barrier();
    Frags f0, f1;
    load(st[0], 0, wave, lane, f0);
    const int nkp = (nk + NS - 1) / NS * NS;
    int knext = kbeg + NS * BK;  // k of the next tile to copy
    auto issue = [&](char* stage) {
      ca.issue(A, knext, klimA, stage, wave);
      cb.issue(B, knext, klimB, stage + kABytes, wave);
      knext += BK;
    };
    for (int t = 0; t < nkp; t += NS) {
      ktile<0>(st, wave, lane, acc, f0, f1, issue);
      ktile<1 % NS>(st, wave, lane, acc, f0, f1, issue);
      if constexpr (NS >= 3) ktile<2 % NS>(st, wave, lane, acc, f0, f1, issue);
      if constexpr (NS >= 4) ktile<3 % NS>(st, wave, lane, acc, f0, f1, issue);
    }
    wait_vmcnt<0>();                      // the copies past the end (zeros) have landed
    __builtin_amdgcn_s_waitcnt(0xC07F);   // and this wave's last (unused) fragment reads
    __builtin_amdgcn_s_barrier();         // before anyone reuses the stages
  }

  // ---- ping-pong schedule (8 waves) ----
  // Waves 0-3 and 4-7 form two groups; waves w and w + 4 share a SIMD.  Every k-tile is one
  // memory phase (this group's copies of the tile NS - 1 ahead, then all of the tile's
  // fragments read into registers) and one compute phase (the tile's products, registers
  // only).  Group 1 runs one phase behind group 0, so that on every SIMD one wave issues
  // products while the other moves data; a barrier ends every phase.  The stage refilled in
  // a memory phase is the one both groups read in the two phases before it.
  __device__ static __forceinline__ void phase_barrier() {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
  }

  template <int S, class Issue>
  __device__ static __forceinline__ void pp_tile(char* const (&st)[NS], int wave, int lane, f32x16 (&acc)[FR][FC],
                                                 Frags (&f)[KK], Issue&& issue) {
    issue(st[(S + NS - 1) % NS]);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) load(st[S], kk, wave, lane, f[kk]);
    // this group's copies up to the next tile have landed (NS - 2 newer tiles may still be in
    // flight); its reads of stage S are done before anyone refills it
    wait_vmcnt<(NS - 2) * CPW>();
    __builtin_amdgcn_s_waitcnt(0xC07F);
    phase_barrier();
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) mma(f[kk], acc);
    phase_barrier();
  }

  // Same contract as run (all kThreads threads call; barriers inside), ping-pong schedule.
  template <bool ZERO = true>
  __device__ static __forceinline__ void run_pp(const GOp& A, const GOp& B, int row0, int col0, int kbeg, int kend,
                                                char* const (&st)[NS], f32x16 (&acc)[FR][FC]) {
    static_assert(NW == 8 && NS >= 3, "two groups of four waves, at least three stages");
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    if constexpr (ZERO) zero(acc);
    const int nk = (kend - kbeg + BK - 1) / BK;
    if (nk <= 0) return;
    const int klimA = min(A.kmax, kend), klimB = min(B.kmax, kend);
    CA ca;
    CB cb;
    if constexpr (BUF) {
      ca.init(A, row0, wave, lane, kbeg, klimA);
      cb.init(B, col0, wave, lane, kbeg, klimB);
    } else {
      ca.init(A, row0, wave, lane);
      cb.init(B, col0, wave, lane);
    }
    int knext = kbeg;  // k of the next tile to copy
    auto issue = [&](char* stage) {
      ca.issue(A, knext, klimA, stage, wave);
      cb.issue(B, knext, klimB, stage + kABytes, wave);
      knext += BK;
    };
    __builtin_amdgcn_s_barrier();  // previous users of the stages are done
#pragma unroll
    for (int s = 0; s < NS - 1; ++s) issue(st[s]);
    wait_vmcnt<(NS - 2) * CPW>();  // tile 0
    __builtin_amdgcn_s_barrier();
    const bool lag = wave >= 4;
    if (lag) phase_barrier();  // group 1 starts one phase behind
    Frags f[KK];
    const int nkp = (nk + NS - 1) / NS * NS;
    for (int t = 0; t < nkp; t += NS) {
      pp_tile<0>(st, wave, lane, acc, f, issue);
      pp_tile<1>(st, wave, lane, acc, f, issue);
      pp_tile<2 % NS>(st, wave, lane, acc, f, issue);
      if constexpr (NS >= 4) pp_tile<3 % NS>(st, wave, lane, acc, f, issue);
    }
    if (!lag) phase_barrier();  // the barrier group 1 took at the start
    wait_vmcnt<0>();                      // the copies past the end (zeros) have landed
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_s_barrier();         // before anyone reuses the stages
  }

  struct ZeroInit {
    __device__ __forceinline__ void operator()(int, f32x16 (&acc)[FR][FC]) const { zero(acc); }
  };
  // A sequence of ntiles output tiles over k in [0, K): tile i uses A rows from
  // row0 + i * BR and the same B rows (col0).  One copy pipeline runs through the tile
  // boundaries; epi(i, acc) is called after tile i's last product, while the next tile's
  // copies are in flight, and must not touch the LDS stages.  init(i, acc) sets the
  // accumulators before tile i's first product (zero by default; a caller can start them
  // at a per-row offset, which then enters the sum exactly as an fp32 addend).  No row
  // gather on A.
  template <class Epi, class Init = ZeroInit>
  __device__ static __forceinline__ void run_seq(const GOp& A, const GOp& B, int row0, int col0, int ntiles, int K,
                                                 char* const (&st)[NS], f32x16 (&acc)[FR][FC], Epi&& epi,
                                                 Init&& init = Init{}) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: copy targets in scalar registers
    if (ntiles > 0) init(0, acc);
    else zero(acc);
    const int nk = (K + BK - 1) / BK;
    if (nk <= 0 || ntiles <= 0) return;
    const int klimA = min(A.kmax, K), klimB = min(B.kmax, K);
    CA ca;
    CB cb;
    if constexpr (BUF) {
      ca.init(A, row0, wave, lane, 0, klimA);
      cb.init(B, col0, wave, lane, 0, klimB);
    } else {
      ca.init(A, row0, wave, lane);
      cb.init(B, col0, wave, lane);
    }
    int ctile = 0, ck = 0;  // copy stream position
    auto issue = [&](char* stage) {
      if (ck == nk) {
        ck = 0;
        ++ctile;
        ca.retarget(A, row0 + ctile * BR, wave, lane);
      }
      const bool live = ctile < ntiles;
      ca.issue(A, ck * BK, live ? klimA : 0, stage, wave);
      cb.issue(B, ck * BK, live ? klimB : 0, stage + kABytes, wave);
      ++ck;
    };
    __builtin_amdgcn_s_barrier();
#pragma unroll
    for (int s = 0; s < NS; ++s) issue(st[s]);
    wait_vmcnt<(NS - 1) * CPW>();
    __builtin_amdgcn_s_barrier();
    Frags f0, f1;
    load(st[0], 0, wave, lane, f0);
    const int total = ntiles * nk;
    const int totalp = (total + NS - 1) / NS * NS;
    int tile = 0, kt = 0;  // compute stream position
    auto after = [&]() {
      if (++kt == nk) {
        if (tile < ntiles) epi(tile, acc);
        if (tile + 1 < ntiles) init(tile + 1, acc);
        else zero(acc);
        kt = 0;
        ++tile;
      }
    };
    for (int g = 0; g < totalp; g += NS) {
      ktile<0>(st, wave, lane, acc, f0, f1, issue);
      after();
      ktile<1 % NS>(st, wave, lane, acc, f0, f1, issue);
      after();
      if constexpr (NS >= 3) {
        ktile<2 % NS>(st, wave, lane, acc, f0, f1, issue);
        after();
      }
      if constexpr (NS >= 4) {
        ktile<3 % NS>(st, wave, lane, acc, f0, f1, issue);
        after();
      }
    }
    wait_vmcnt<0>();
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_s_barrier();
  }

  // run_seq for K a multiple of NS BK (every tile starts at stage 0, no padded k-tiles) with
  // zero-initialised tiles and an epilogue that issues exactly EXTRA vector memory
  // instructions per wave (stores; epi may use LDS outside the stages).  The first NS - 1
  // k-tiles of the next tile wait with EXTRA more outstanding (the stores were issued after
  // the copies those waits are for), so the stores drain under that tile's first products.
  // The tile loop is nested with each tile's first k-tile group written out, so that the
  // compiler, which waits on its own before reading a stage whose copy it cannot prove has
  // landed, sees the issue order these waits rely on.
  template <int EXTRA, class Epi>
  __device__ static __forceinline__ void run_seq_aligned(const GOp& A, const GOp& B, int row0, int col0, int ntiles,
                                                         int K, char* const (&st)[NS], f32x16 (&acc)[FR][FC],
                                                         Epi&& epi) {
    static_assert(BUF, "buffer-resource copies");
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    zero(acc);
    const int nk = K / BK;  // the caller guarantees K % (NS BK) == 0
    if (nk <= 0 || ntiles <= 0) return;
    const int klimA = min(A.kmax, K), klimB = min(B.kmax, K);
    CA ca;
    CB cb;
    ca.init(A, row0, wave, lane, 0, klimA);
    cb.init(B, col0, wave, lane, 0, klimB);
    int ctile = 0, ck = 0;  // copy stream position
    auto issue = [&](char* stage) {
      if (ck == nk) {
        ck = 0;
        ++ctile;
        ca.retarget(A, row0 + ctile * BR, wave, lane);
      }
      const bool live = ctile < ntiles;
      ca.issue(A, ck * BK, live ? klimA : 0, stage, wave);
      cb.issue(B, ck * BK, live ? klimB : 0, stage + kABytes, wave);
      ++ck;
    };
    __builtin_amdgcn_s_barrier();
#pragma unroll
    for (int s = 0; s < NS; ++s) issue(st[s]);
    wait_vmcnt<(NS - 1) * CPW>();
    __builtin_amdgcn_s_barrier();
    Frags f0, f1;
    load(st[0], 0, wave, lane, f0);
    const int ng = nk / NS;
    auto group = [&]() {
      ktile<0>(st, wave, lane, acc, f0, f1, issue);
      ktile<1 % NS>(st, wave, lane, acc, f0, f1, issue);
      if constexpr (NS >= 3) ktile<2 % NS>(st, wave, lane, acc, f0, f1, issue);
      if constexpr (NS >= 4) ktile<3 % NS>(st, wave, lane, acc, f0, f1, issue);
    };
    auto relaxed_group = [&]() {
      ktile<0, EXTRA>(st, wave, lane, acc, f0, f1, issue);
      if constexpr (NS == 2) {
        ktile<1>(st, wave, lane, acc, f0, f1, issue);
      } else {
        ktile<1, EXTRA>(st, wave, lane, acc, f0, f1, issue);
        if constexpr (NS == 3) ktile<2>(st, wave, lane, acc, f0, f1, issue);
        if constexpr (NS >= 4) {
          ktile<2, EXTRA>(st, wave, lane, acc, f0, f1, issue);
          ktile<3>(st, wave, lane, acc, f0, f1, issue);
        }
      }
    };
    group();
    for (int gi = 1; gi < ng; ++gi) group();
    epi(0, acc);
    zero(acc);
    for (int t = 1; t < ntiles; ++t) {
      relaxed_group();
      for (int gi = 1; gi < ng; ++gi) group();
      epi(t, acc);
      zero(acc);
    }
    wait_vmcnt<0>();
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_s_barrier();
  }
};

// 8-wave 256 x 256 tile of C = A B^T for a k-contiguous A whose rows lie far apart (the dH
// product's dZ rows) and a row-contiguous B, on the ping-pong schedule.  A is copied 64 deep, so
// that every row piece is a whole 128-byte line (a 32-deep copy takes half lines, which cost
// the cache about as much as whole ones): two 32 KB A super-stages (k-tiles 2j, 2j + 1); B 32
// deep in four 16 KB stages.  Each super-stage is refilled in the memory phase of an even
// k-tile, two k-tiles before it is read; B is copied three k-tiles ahead.  Every stage is an
// LDS array of its own, so that the compiler can tell the stage being read from the ones being
// filled (it waits for every copy in flight before a read it cannot tell apart from them).
template <int WR, int WC>
struct GemmA64 : Gemm<256, 256, 32, LL::KC, LL::MC, 4, WR, WC, true> {
  using Base = Gemm<256, 256, 32, LL::KC, LL::MC, 4, WR, WC, true>;
  using Frags = typename Base::Frags;
  using CA = TileCopy<LL::KC, 256, 64, 8, true>;
  using CB = typename Base::CB;
  static constexpr int FR = Base::FR, FC = Base::FC, KK = Base::KK;
  static constexpr int CPA = CA::kPerWave, CPB = CB::kPerWave;
  static_assert(Base::NW == 8 && CA::kBytes == 32768 && CB::kBytes == 16384, "stage sizes");
  static_assert(2 * CPB + CPA < 64, "vmcnt range");

  // sl[0], sl[1]: A super-stages; sl[2..5]: B stages
  template <int S>
  __device__ static __forceinline__ void load_tile(char* const (&sl)[6], int wave, int lane, Frags (&f)[KK]) {
    const int wr0 = (wave / WC) * (256 / WR), wc0 = (wave % WC) * (256 / WC);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
      for (int i = 0; i < FR; ++i)
        f[kk].a[i] = frag<LL::KC, 256, 64>(sl[S / 2], wr0 + 32 * i, (S % 2) * 32 + kk * 16, lane);
#pragma unroll
      for (int j = 0; j < FC; ++j) f[kk].b[j] = frag<LL::MC, 256, 32>(sl[2 + S], wc0 + 32 * j, kk * 16, lane);
    }
  }

  template <int S, class IssueA, class IssueB>
  __device__ static __forceinline__ void pp_tile(char* const (&sl)[6], int wave, int lane, f32x16 (&acc)[FR][FC],
                                                 Frags (&f)[KK], IssueA&& issue_a, IssueB&& issue_b) {
    // even k-tile t: the A super-stage of k-tiles t - 2, t - 1 takes k-tiles t + 2, t + 3
    if constexpr (S % 2 == 0) issue_a(sl[(S / 2 + 1) % 2]);
    issue_b(sl[2 + (S + 3) % 4]);  // k-tile t + 3 into the stage of t - 1
    load_tile<S>(sl, wave, lane, f);
    // the next k-tile's copies from this wave have landed: B's (issued three k-tiles back) and,
    // after an odd k-tile, the A super-stage issued in the previous (even) k-tile, before that
    // k-tile's B copy; what may still be in flight was issued after them
    if constexpr (S % 2 == 0) wait_vmcnt<2 * CPB + CPA>();
    else wait_vmcnt<2 * CPB>();
    __builtin_amdgcn_s_waitcnt(0xC07F);
    Base::phase_barrier();
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) Base::mma(f[kk], acc);
    Base::phase_barrier();
  }

  // Same contract as Gemm::run (all 512 threads call; barriers inside), stages declared here.
  template <bool ZERO = true>
  __device__ static __forceinline__ void product(const GOp& A, const GOp& B, int row0, int col0, int kbeg, int kend,
                                                 f32x16 (&acc)[FR][FC]) {
    __shared__ __attribute__((aligned(1024))) char a0[32768], a1[32768];
    __shared__ __attribute__((aligned(1024))) char b0[16384], b1[16384], b2[16384], b3[16384];
    char* const sl[6] = {a0, a1, b0, b1, b2, b3};
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    if constexpr (ZERO) Base::zero(acc);
    const int nk = (kend - kbeg + 31) / 32;
    if (nk <= 0) return;
    const int klimA = min(A.kmax, kend), klimB = min(B.kmax, kend);
    CA ca;
    CB cb;
    ca.init(A, row0, wave, lane, kbeg, klimA);
    cb.init(B, col0, wave, lane, kbeg, klimB);
    int kna = kbeg, knb = kbeg;  // k of the next A super-tile and B tile to copy
    auto issue_a = [&](char* stage) {
      ca.issue(A, kna, klimA, stage, wave);
      kna += 64;
    };
    auto issue_b = [&](char* stage) {
      cb.issue(B, knb, klimB, stage, wave);
      knb += 32;
    };
    __builtin_amdgcn_s_barrier();  // previous users of the stages are done
    issue_a(sl[0]);
#pragma unroll
    for (int b = 0; b < 3; ++b) issue_b(sl[2 + b]);
    wait_vmcnt<2 * CPB>();  // A super-tile 0 and B tile 0
    __builtin_amdgcn_s_barrier();
    const bool lag = wave >= 4;
    if (lag) Base::phase_barrier();  // group 1 starts one phase behind
    Frags f[KK];
    const int nkp = (nk + 3) / 4 * 4;
    for (int t = 0; t < nkp; t += 4) {
      pp_tile<0>(sl, wave, lane, acc, f, issue_a, issue_b);
      pp_tile<1>(sl, wave, lane, acc, f, issue_a, issue_b);
      pp_tile<2>(sl, wave, lane, acc, f, issue_a, issue_b);
      pp_tile<3>(sl, wave, lane, acc, f, issue_a, issue_b);
    }
    if (!lag) Base::phase_barrier();
    wait_vmcnt<0>();
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_s_barrier();
  }
};

// 8-wave 256 x 256 tile runs of C = A B^T with epilogues (the contract of
// Gemm::run_seq_aligned, K a multiple of 128) for a k-contiguous A whose 64-byte row pieces
// would be half cache lines (W rows of 1 KB and more) and a row-contiguous B, on the interleaved
// schedule.  A is copied 64 deep, so that every row piece is a whole 128-byte line: two 32 KB A
// super-stages (k-tiles 2j, 2j + 1) and four 16 KB B stages, each an LDS array of its own
// (declared here; the compiler waits for every copy in flight before a read of an array it
// cannot tell apart from one being filled).  After the barrier that ends k-tile t, B's stage of
// t takes t + 4 and, for odd t, the A super-stage of t - 1, t takes t + 3, t + 4 (read two
// k-tiles later); the copies of A (odd t) are issued before B's, and the prologue issues in the
// same order (A0 B0 B1 B2 A1 B3), so every k-tile waits by the same count.
template <int WR, int WC>
struct GemmMidA64 : Gemm<256, 256, 32, LL::KC, LL::MC, 4, WR, WC, true> {
  using Base = Gemm<256, 256, 32, LL::KC, LL::MC, 4, WR, WC, true>;
  using Frags = typename Base::Frags;
  using CA = TileCopy<LL::KC, 256, 64, 8, true>;
  using CB = typename Base::CB;
  static constexpr int FR = Base::FR, FC = Base::FC, KK = Base::KK, NM = Base::NM;
  static constexpr int CPA = CA::kPerWave, CPB = CB::kPerWave;
  static constexpr int kKernelStageBytes = 16;
  static_assert(Base::NW == 8 && CA::kBytes == 32768 && CB::kBytes == 16384 && KK == 2, "layout");
  static_assert(3 * CPB + CPA + 16 < 64, "vmcnt range");

  // fragments of k-step kk of k-tile t (S = t mod 4)
  template <int S>
  __device__ static __forceinline__ void load(char* const (&sl)[6], int kk, int wave, int lane, Frags& f) {
    const int wr0 = (wave / WC) * (256 / WR), wc0 = (wave % WC) * (256 / WC);
#pragma unroll
    for (int i = 0; i < FR; ++i) f.a[i] = frag<LL::KC, 256, 64>(sl[S / 2], wr0 + 32 * i, (S % 2) * 32 + kk * 16, lane);
#pragma unroll
    for (int j = 0; j < FC; ++j) f.b[j] = frag<LL::MC, 256, 32>(sl[2 + S], wc0 + 32 * j, kk * 16, lane);
  }

  // k-tile t (S = t mod 4); the fragments of its first k-step are in f0.  XTRA: as in
  // Gemm::ktile (an epilogue's stores were issued after the copies this wait is for).
  template <int S, int XTRA = 0, class IssueA, class IssueB>
  __device__ static __forceinline__ void ktile(char* const (&sl)[6], int wave, int lane, f32x16 (&acc)[FR][FC],
                                               Frags& f0, Frags& f1, IssueA&& issue_a, IssueB&& issue_b) {
    constexpr int NH = NM / 2;
    load<S>(sl, 1, wave, lane, f1);
    Base::mma(f0, acc);
    Base::template interleave<0>();
    Base::template mma_range<0, NH>(f1, acc);
    // k-tile t + 1 has landed: B's copy (issued after k-tile t - 3) and, for odd t, the A
    // super-stage (issued after k-tile t - 2, before that k-tile's B copy)
    if constexpr (S % 2 == 0) wait_vmcnt<2 * CPB + CPA + XTRA>();
    else wait_vmcnt<2 * CPB + XTRA>();
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's reads of k-tile t are done
    __builtin_amdgcn_s_barrier();
    if constexpr (S % 2 == 1) issue_a(sl[S / 2]);  // the super-stage of t - 1, t
    issue_b(sl[2 + S]);
    load<(S + 1) % 4>(sl, 0, wave, lane, f0);
    Base::template mma_range<NH, NM>(f1, acc);
    Base::template interleave<(S % 2 == 1) ? CPA + CPB : CPB, NM - NH>();
  }

  // The stage arrays, one set per kernel (not per seq_aligned instantiation).
  __device__ static __forceinline__ void stages(char* (&sl)[6]) {
    __shared__ __attribute__((aligned(1024))) char a0[32768], a1[32768];
    __shared__ __attribute__((aligned(1024))) char b0[16384], b1[16384], b2[16384], b3[16384];
    sl[0] = a0;
    sl[1] = a1;
    sl[2] = b0;
    sl[3] = b1;
    sl[4] = b2;
    sl[5] = b3;
  }

  template <int EXTRA, class Epi>
  __device__ static __forceinline__ void seq_aligned(const GOp& A, const GOp& B, int row0, int col0, int ntiles,
                                                     int K, f32x16 (&acc)[FR][FC], Epi&& epi) {
    char* sl[6];
    stages(sl);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    Base::zero(acc);
    const int nk = K / 32;  // the caller guarantees K % 128 == 0
    if (nk <= 0 || ntiles <= 0) return;
    const int klimA = min(A.kmax, K), klimB = min(B.kmax, K);
    CA ca;
    CB cb;
    ca.init(A, row0, wave, lane, 0, klimA);
    cb.init(B, col0, wave, lane, 0, klimB);
    int atile = 0, ak = 0, btile = 0, bk = 0;  // copy stream positions (output tile, k)
    auto issue_a = [&](char* stage) {
      if (ak == K) {
        ak = 0;
        ++atile;
        ca.retarget(A, row0 + atile * 256, wave, lane);
      }
      ca.issue(A, ak, atile < ntiles ? klimA : 0, stage, wave);
      ak += 64;
    };
    auto issue_b = [&](char* stage) {
      if (bk == K) {
        bk = 0;
        ++btile;
      }
      cb.issue(B, bk, btile < ntiles ? klimB : 0, stage, wave);
      bk += 32;
    };
    __builtin_amdgcn_s_barrier();
    issue_a(sl[0]);
    issue_b(sl[2]);
    issue_b(sl[3]);
    issue_b(sl[4]);
    issue_a(sl[1]);
    issue_b(sl[5]);
    wait_vmcnt<3 * CPB + CPA>();  // A super-tile 0 and B tile 0
    __builtin_amdgcn_s_barrier();
    Frags f0, f1;
    load<0>(sl, 0, wave, lane, f0);
    const int ng = nk / 4;
    auto group = [&]() {
      ktile<0>(sl, wave, lane, acc, f0, f1, issue_a, issue_b);
      ktile<1>(sl, wave, lane, acc, f0, f1, issue_a, issue_b);
      ktile<2>(sl, wave, lane, acc, f0, f1, issue_a, issue_b);
      ktile<3>(sl, wave, lane, acc, f0, f1, issue_a, issue_b);
    };
    auto relaxed_group = [&]() {
      ktile<0, EXTRA>(sl, wave, lane, acc, f0, f1, issue_a, issue_b);
      ktile<1, EXTRA>(sl, wave, lane, acc, f0, f1, issue_a, issue_b);
      ktile<2, EXTRA>(sl, wave, lane, acc, f0, f1, issue_a, issue_b);
      ktile<3>(sl, wave, lane, acc, f0, f1, issue_a, issue_b);
    };
    group();
    for (int gi = 1; gi < ng; ++gi) group();
    epi(0, acc);
    Base::zero(acc);
    for (int t = 1; t < ntiles; ++t) {
      relaxed_group();
      for (int gi = 1; gi < ng; ++gi) group();
      epi(t, acc);
      Base::zero(acc);
    }
    wait_vmcnt<0>();
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_s_barrier();
  }
};

}  // namespace bf
}  // namespace pctc
