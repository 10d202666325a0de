// Host-side declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "pctc_device.h"

namespace pctc {

// Kernel timing: records a start event on construction and a stop event on destruction
// when timing is enabled (pctc_prof_enable); the scope owns its two events until it closes,
// when the pair joins the shared list that is resolved when the totals are read (a reader in
// another thread meanwhile neither sees nor recycles them).  prof_flush(), at the end of each
// entry point, resolves that list only once it is long.
struct Prof {
  Prof(const char* name, hipStream_t stream);
  ~Prof();
  const char* name;
  hipEvent_t start = nullptr, stop = nullptr;
  hipStream_t stream;
};
void prof_flush();

constexpr int kDefaultChunk = 16384;
constexpr float kKeepSlack = 1e-3f;  // nats added to the beam threshold (tie/rounding rule)

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ---- union / relabel -------------------------------------------------------------------
// u_ids[remap[v]] = v for remap[v] >= 0 and K = 1 + max remap (K zeroed here).
hipError_t launch_remap_invert(const int32_t* remap, int32_t V, int32_t* u_ids, int32_t* K, hipStream_t stream);
// scratch: union_scratch_bytes(V) (a membership bitmap and a count per block of classes).
size_t union_scratch_bytes(int32_t V);
hipError_t launch_union_remap(const int32_t* targets, int32_t total, int32_t blank, int32_t V,
                              int32_t* remap, int32_t* u_ids, int32_t* y_rel, int32_t* K, int32_t* err,
                              void* scratch, hipStream_t stream);

// ---- normaliser and selected log-probabilities ------------------------------------------
int lse_partitions(int M, int V);
// Heads with D >= kWideD run their bf16 products on 8-wave 256 x 256 tiles.
constexpr int kWideD = 2048;
// Most vocabulary partitions of a normaliser or argmax launch (partial buffer rows): 256,
// or kMaxLseParts for wide heads (one vocabulary tile per workgroup there).
constexpr int kMaxLseParts = 1024;
inline int lse_max_parts(int D) { return D >= kWideD ? kMaxLseParts : 256; }
size_t lse_partial_bytes(int M, int D);
// bias: device float [V] or null (logits H W^T + b).
hipError_t launch_lse(int dtype, const void* H, int M, int D, const void* W, const float* bias, int V,
                      float2* partials, double* lam, float2* lam2, hipStream_t stream);
// The same in two halves: the partial (max, sum) pairs over the vocabulary partitions
// (P_out: partitions written), then lambda and its hi/lo pair from them; with Zd the second
// half also writes S[m * ldS + j] = float(Zd[m * ldS + j] - lambda_m) for j < *K.
hipError_t launch_lse_partials(int dtype, const void* H, int M, int D, const void* W, const float* bias, int V,
                               float2* partials, int* P_out, hipStream_t stream);
// With g (forecast dense-part factors), also rowscale[m] = -g_m exp(-lambda_m) and *einv = 1
// if any lambda_m lies outside [kEMin, kEMax] (the normaliser's E = exp(z) is then unusable:
// bf16 overflow or significant underflow).
constexpr double kEMin = -40.0, kEMax = 60.0;
hipError_t launch_lse_finalize(const float2* partials, int M, int P, double* lam, float2* lam2, const double* Zd,
                               const int32_t* K, float* S, int ldS, hipStream_t stream, const float* g = nullptr,
                               float* rowscale = nullptr, int32_t* einv = nullptr);
hipError_t launch_gather_s(int dtype, const void* H, int M, int D, const void* W, const float* bias,
                           const int32_t* u_ids, const int32_t* K, int K_max, const double* lam, float* S, int ldS,
                           hipStream_t stream);

// ---- greedy emission head -----------------------------------------------------------------
// partials: lse_partial_bytes(M, D); ids [M]; tokens [M] (utterance n at toff[n]); lengths [N].
hipError_t launch_greedy(int dtype, const void* H, int M, int D, const void* W, const float* bias, int V,
                         const int32_t* toff, int N, int blank, float2* partials, int32_t* ids, int32_t* tokens,
                         int32_t* lengths, hipStream_t stream);
hipError_t launch_amax_partial_bf16(const uint16_t* H, int M, int D, const uint16_t* W, const float* bias, int V,
                                    float2* partials, int* P_out, hipStream_t stream);

// A second operand set for a dW product's launch: out[v][:] = sum over frames of Z[m][v] Hs[m][:]
// for v < cols (cut to 2 *kdev when kdev is set), Z [M][ld] bf16.  The union columns' dW_u
// rides this way in the last chunk's dense dW launch (its work fits the launch's last round).
struct DwExtra {
  const uint16_t* Z = nullptr;  // null: none
  int ld = 0, cols = 0;
  const int32_t* kdev = nullptr;
  float* out = nullptr;
  hipEvent_t ready = nullptr;   // recorded once Z is written (second stream); waited on first
};

// ---- backward ---------------------------------------------------------------------------
struct BwdPlan {
  int chunk;       // vocabulary columns per step
  int splits;      // k-slices of the dH product per chunk
  int Mp;          // padded frame count (pitch of the transposed head input)
  // hst_bytes: Hs transposed, [D][Mp] bf16, read by the dense recompute of narrow bf16 heads
  size_t dz_bytes, ht_bytes, part_bytes, lam2_bytes, dbpart_bytes, hst_bytes, total;
};
BwdPlan plan_bwd(int dtype, int M, int D, int V, int chunk);
// Column multiple of the default chunk of narrow bf16 heads: the normaliser's partition width
// (eight 256-row tiles; any V up to PCTC_MAX_VOCAB keeps it within 256 partitions).
constexpr int kEAlign = 2048;
// The bf16 fused schedule's side of the recomputed backward.  With a second stream: work i
// (i < nwork) is enqueued on that stream after chunk i + 1 of the dense part (the caller's
// stream records gate[i], the second stream waits for it, then work[i].fn(work[i].ctx)
// enqueues), or at the last chunk's dH product when there are fewer chunks, so that the
// second stream's kernels run beside the next chunk's recompute, whose many short workgroups
// leave room for them, rather than hold compute units while a dH or dW product launches.
// The last chunk records dh_done after its dH product; the second stream waits for it and
// runs the final dH reduction (adding dH_extra, written by its work) beside the chunk's dW
// product, then records reduced, which the caller's stream waits for before the call returns.
// When the dense part accumulates dH in place (a single split-K slice: no partial buffer),
// after_dh runs there instead of the reduction (it adds the union columns' part to dH).
// hs_built: the masked copy of H (bwd_hs) was already written, from the same g, on a stream
// the caller's stream has waited for.  udw (when udw.Z is set): with dH wanted, the last
// chunk's dW launch waits for udw.ready and also computes the union columns' dW_u.
struct SideWork {
  hipError_t (*fn)(void*) = nullptr;
  void* ctx = nullptr;
};
struct BwdSide {
  hipStream_t stream = nullptr;
  hipEvent_t gate[2] = {nullptr, nullptr};
  hipEvent_t dh_done = nullptr, reduced = nullptr;
  SideWork work[2];
  SideWork after_dh;
  // enqueued on the second stream once the first chunk's dH product is (beside that chunk's dW),
  // before the works; front_gate orders it after everything enqueued on the caller's stream
  SideWork front;
  hipEvent_t front_gate = nullptr;
  int nwork = 0;
  const float* dH_extra = nullptr;
  bool hs_built = false;
  DwExtra udw;  // the union columns' dW_u, folded into the last chunk's dW launch (dH wanted)
  const struct ChunkE* ce = nullptr;  // the first chunk's dZ rows come from the normaliser
};
// the masked copy of H (rows of frames with g == 0 zeroed) inside the backward's scratch, and
// its transpose [D][Mp] (null where the plan has none)
uint16_t* bwd_hs(void* scratch, const BwdPlan& plan);
uint16_t* bwd_hst(void* scratch, const BwdPlan& plan);
// S/ldS: the forward's selected log-probabilities (the bf16 path writes the union columns
// of each recomputed chunk from them).  remap == null (bf16 path): the dense part -g p only.
hipError_t launch_head_bwd(int dtype, const void* H, int M, int D, const void* W, const float* bias, int V,
                           const float2* lam2, const float* G, int ldG, const float* g, const int32_t* remap,
                           const float* S, int ldS, float* dH, float* dW, float* db, void* scratch,
                           const BwdPlan& plan, hipStream_t stream, const BwdSide* side = nullptr);
hipError_t launch_lam2(const double* lam, int M, float2* lam2, hipStream_t stream);

// ---- bf16 kernels on the direct-to-LDS engine (head_gemm_bf16.hip) ---------------------
hipError_t launch_lse_partial_bf16(const uint16_t* H, int M, int D, const uint16_t* W, const float* bias, int V,
                                   float2* partials, int* P_out, hipStream_t stream);
// Zd (may be null): write the selected logits in double (Zd[m * ldS + j]) instead of S; lam
// is then not read (launch_lse_finalize subtracts it).
hipError_t launch_gather_s_bf16(const uint16_t* H, int M, int D, const uint16_t* W, const float* bias,
                                const int32_t* u_ids, const int32_t* K, int K_max, const double* lam, float* S, int ldS,
                                hipStream_t stream, double* Zd = nullptr);
// One chunk of the recomputed backward: the recompute of dZ (when `recompute`), then the dH
// and dW products it feeds.
// The backward's first chunk when the normaliser wrote its dZ rows as E = exp(z) without the
// per-frame factor s_m = -g_m exp(-lambda_m) (bf16 fused schedule, narrow heads): the dH
// product scales its rows by rowscale and the dW product reads Hp = s Hs instead of Hs; the
// recompute runs only when *einv is set (E unusable; rowscale then holds ones and Hp a copy
// of Hs).
struct ChunkE {
  const float* rowscale = nullptr;
  const uint16_t* Hp = nullptr;
  const int32_t* einv = nullptr;
};
hipError_t launch_bwd_chunk_bf16(const uint16_t* Hs, int M, int D, const uint16_t* W, const float* bias, int c0,
                                 int cw, const float2* lam2, const float* G, int ldG, const float* g,
                                 const int32_t* remap, const float* S, int ldS, uint16_t* dZ, int chunk, float* part,
                                 int slice, bool recompute, bool want_dH, bool want_dW, float* dW, float* db,
                                 float* dbpart, hipStream_t stream, const DwExtra* extra = nullptr,
                                 const ChunkE* ce = nullptr, const uint16_t* Hst = nullptr, int Mp = 0);
// Partitions of the normaliser that can write E for a first chunk of `chunk` columns (0: none;
// narrow heads with D a multiple of 128, chunk a multiple of the partition width).
int lse_e_parts_bf16(int M, int D, int V, int chunk);
// The normaliser (no bias) that also writes E = exp(z) in bf16 at E[m * epitch + v] for the
// rows of its first eparts partitions, and clears *einv (see launch_lse_finalize).  With Ht
// (H transposed, [D][Mp], from launch_ht_build_bf16) the frames are read from there.
hipError_t launch_lse_partial_e_bf16(const uint16_t* H, int M, int D, const uint16_t* W, int V, float2* partials,
                                     int* P_out, uint16_t* E, int epitch, int eparts, int32_t* einv,
                                     hipStream_t stream, const uint16_t* Ht = nullptr, int Mp = 0);
// rowscale/Hp of ChunkE from the finalize's s_m (in rowscale) and its check flag.
hipError_t launch_hs_scale_bf16(const uint16_t* Hs, int M, int D, const int32_t* einv, float* rowscale, uint16_t* Hp,
                                hipStream_t stream);
// Union-column part of the backward (bf16 path): dH_u = G W_U written into dH [M][D] (which
// the final reduction then adds the dense part to), or later added to dH, and into its own
// buffers dW_u = G^T H [K_max][D] and db_u = column sums of G [K_max], frames with g == 0 left
// out; then union_merge adds dW_u, db_u into the rows U of dW, db.  scratch:
// union_corr_bytes().  Hs: H with the rows of frames with g == 0 zeroed (the dense part's
// copy, bwd_hs), needed for dW_u.
// Gb [M][2 ldK] bf16 (union_gb_bytes): the [hi | lo] copy of G, caller-placed.  dh_later: dH_u is
// not formed here but by launch_union_dh_bf16, which adds it to dH (after the dense part).
// dw_elsewhere: dW_u's buffer is sized and merged as usual, but its product is left to a dense
// dW launch (union_dw_extra gives that launch's second operand set).
size_t union_corr_bytes(int M, int D, int K_max, bool want_dW);
size_t union_gb_bytes(int M, int K_max);
hipError_t launch_union_part_bf16(const float* G, int ldG, const int32_t* Kdev, int K_max, const int32_t* u_ids,
                                  const uint16_t* W, const uint16_t* Hs, int M, int D, float* dH, bool dh_later,
                                  bool want_dW, bool want_db, void* scratch, uint16_t* Gb, hipStream_t stream,
                                  bool dw_elsewhere = false);
DwExtra union_dw_extra(int M, int D, int K_max, const int32_t* Kdev, void* scratch, const uint16_t* Gb);
hipError_t launch_union_dh_bf16(const uint16_t* Gb, const int32_t* Kdev, int K_max, int M, int D, float* dH,
                                void* scratch, bool want_dW, hipStream_t stream);
hipError_t launch_union_merge_bf16(const int32_t* Kdev, int K_max, const int32_t* u_ids, int M, int D, float* dW,
                                   float* db, void* scratch, hipStream_t stream);
hipError_t launch_hs_build_bf16(const uint16_t* H, int M, int D, const float* g, uint16_t* Hs, hipStream_t stream);
// Ht[d][m] = H[m][d] ([D][Mp], Mp a multiple of 64; frames with g[m] == 0 zeroed when g is
// given; columns m >= M zero), and with Hs given the masked rows in H's layout as well.
hipError_t launch_ht_build_bf16(const uint16_t* H, int M, int D, const float* g, uint16_t* Hs, uint16_t* Ht, int Mp,
                                hipStream_t stream);

// ---- grouped logits for a stock CTC (grouped_head.hip) ----------------------------------
// small: device int32 [2] = {K, error flag}; remap[v] = j for v = u_ids[j], else -1.
hipError_t launch_grouped_index(const int32_t* u_ids, int K, int V, int32_t* remap, int32_t* small,
                                hipStream_t stream);
hipError_t launch_grouped_comp_bias(const float* bias, const int32_t* remap, int V, float* bo, hipStream_t stream);
hipError_t launch_fill_d(double* x, int n, double val, hipStream_t stream);
// logp [M][K + 1]: raw selected logits in, exported log-probabilities out; lam [M] out.
hipError_t launch_grouped_finalize(float* logp, int K, int M, const double* lse_o, double* lam, hipStream_t stream);
hipError_t launch_grouped_adapter(const float* logp, const float* dlogp, int K, int M, float* G, float* g,
                                  hipStream_t stream);

// ---- alignment lattice ------------------------------------------------------------------
struct DpPlan {
  int N, M, Y, Smax;
  bool pruned;
  int64_t lattice;  // sum_n T_n (2U_n+1)
  size_t off_toff, off_yoff, off_soff, off_frame_utt, off_dup_next, off_dup_first, off_logp, off_status,
      off_tab_fa, off_tab_fb, off_tab_va, off_tab_vb, off_sc_fa, off_sc_fb, off_sc_va, off_sc_vb,
      off_vbest, off_mask, off_dummy, total;
};
DpPlan plan_dp(int N, const int32_t* T, const int32_t* U, float beam);
// Uploads the host offsets into the scratch (async) and runs the whole lattice stage.
// weight: device float [N] loss weights of the utterances, or null (all 1): G rows of
// utterance n are -w_n gamma.
// phase: kDpAll, or kDpFront (zeroing of G and g, prep, the Viterbi pass and the arc mask)
// then kDpBack (the log-sum passes and the occupancies, G and g) on the same stream; kDpFront
// may itself be split into kDpPrep (the zeroing and prep, which do not read S) and kDpVit.
constexpr int kDpAll = 0, kDpFront = 1, kDpBack = 2, kDpPrep = 3, kDpVit = 4;
// Longest utterance (frames) whose lattice front the two-stream schedule starts beside the first
// chunk's dW product rather than at once.
constexpr int kFrontDeferT = 512;
hipError_t launch_ctc_dp(const DpPlan& plan, const int32_t* T, const int32_t* U, const float* S, int ldS,
                         const int32_t* y_rel, float beam, const float* weight, double* loss_n, int32_t* status,
                         float* G, float* g, uint8_t* keep_mask_out, void* scratch, int K_max, hipStream_t stream,
                         void* host_staging, int phase = kDpAll);
// delta [nbeams][N]: discarded posterior mass of each utterance at each beam (host beams).
// Needs a plan made with a finite beam (the Viterbi tables and the arc mask).
hipError_t launch_discarded_mass(const DpPlan& plan, const float* S, int ldS, const int32_t* y_rel, const float* beams,
                                 int nbeams, double* delta, void* scratch, int K_max, hipStream_t stream);
hipError_t launch_loss_reduce(int N, const double* loss_n, const int32_t* status, const float* weight, double* loss,
                              hipStream_t stream);
// Forecast of g before the lattice runs: g_pred[m] = -w_n on utterances whose targets fit
// their frames and whose normalisers are finite (and w_n != 0), else 0; pred[n] = 1/0.
// Needs the offsets uploaded into the lattice scratch.
hipError_t launch_g_forecast(const DpPlan& plan, void* scratch, const int32_t* y_rel, const double* lam,
                             const float* weight, float* g_pred, int32_t* pred, hipStream_t stream);
// flag[0] = 1 when the lattice's inclusions differ from the forecast.
hipError_t launch_forecast_check(int N, const int32_t* status, const float* weight, const int32_t* pred,
                                 int32_t* flag, hipStream_t stream);

}  // namespace pctc
