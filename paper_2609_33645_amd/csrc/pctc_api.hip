// C ABI of the Pruned CTC library: argument checks, workspace layout, stage ordering
// (Algorithm 1 of "Pruned CTC for Memory-Efficient Large-Vocabulary ASR Training").
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <functional>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/prunedctc.h"
#include "pctc_internal.h"

namespace pctc {

// ---------------------------------------------------------------------------------------
// Kernel timing
// ---------------------------------------------------------------------------------------
namespace {
struct ProfRec {
  const char* name;
  hipEvent_t start, stop;
};
struct ProfState {
  std::mutex mu;
  bool enabled = false;
  std::string only;  // when non-empty, only kernels of this name are timed
  std::vector<hipEvent_t> pool;
  std::vector<ProfRec> pending;
  std::vector<std::string> names;
  std::map<std::string, std::pair<double, int64_t>> totals;
};
ProfState& prof_state() {
  static ProfState* s = new ProfState();  // never destroyed: events may outlive static teardown
  return *s;
}
hipEvent_t take_event(ProfState& s) {
  if (!s.pool.empty()) {
    hipEvent_t e = s.pool.back();
    s.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
thread_local char g_last_error[512] = "";
}  // namespace

Prof::Prof(const char* nm, hipStream_t st) : name(nm), stream(st) {
  ProfState& s = prof_state();
  if (!s.enabled) return;
  std::lock_guard<std::mutex> lk(s.mu);
  if (!s.only.empty() && s.only != nm) return;
  start = take_event(s);
  stop = take_event(s);
  if (!start || !stop) {
    if (start) s.pool.push_back(start);
    if (stop) s.pool.push_back(stop);
    start = stop = nullptr;
    return;
  }
  hipEventRecord(start, stream);
}

Prof::~Prof() {
  if (!start) return;
  ProfState& s = prof_state();
  std::lock_guard<std::mutex> lk(s.mu);
  hipEventRecord(stop, stream);
  s.pending.push_back(ProfRec{name, start, stop});
}

// Resolves the pending event pairs into the per-kernel totals (s.mu held).
static void prof_resolve(ProfState& s) {
  for (auto& r : s.pending) {
    float ms = 0.f;
    if (hipEventSynchronize(r.stop) == hipSuccess && hipEventElapsedTime(&ms, r.start, r.stop) == hipSuccess) {
      auto it = s.totals.find(r.name);
      if (it == s.totals.end()) {
        s.names.push_back(r.name);
        s.totals[r.name] = {static_cast<double>(ms), 1};
      } else {
        it->second.first += ms;
        it->second.second += 1;
      }
    }
    s.pool.push_back(r.start);
    s.pool.push_back(r.stop);
  }
  s.pending.clear();
}

// Called at the end of every entry point.  The pairs are resolved when the totals are read
// (or reset), so that timing costs a call only its event records; here only a long backlog
// is resolved, which bounds the events held.
void prof_flush() {
  constexpr size_t kMaxPending = 4096;
  ProfState& s = prof_state();
  std::lock_guard<std::mutex> lk(s.mu);
  if (s.pending.size() >= kMaxPending) prof_resolve(s);
}

static void set_error(const char* what, hipError_t e) {
  snprintf(g_last_error, sizeof(g_last_error), "%s: %s", what, hipGetErrorString(e));
}

// ---------------------------------------------------------------------------------------
// Workspace layout
// ---------------------------------------------------------------------------------------
struct Layout {
  int N, M, Y, K_max, ldS;
  bool pruned;
  DpPlan dp;
  BwdPlan bwd;
  size_t o_remap, o_ubits, o_uids, o_yrel, o_small, o_status, o_lossn, o_part, o_lam, o_lam2, o_S, o_G, o_g, o_gpred, o_pred,
      o_corr, o_dp, o_bwd, o_zd, total;
  // narrow bf16 heads: partitions of the normaliser that write the first chunk's E (0: none),
  // the per-frame factors and the scaled H of that chunk's dW product
  int eparts;
  size_t o_escale, o_hp;
  // with E: H transposed [D][Mp] for the normaliser (0: none)
  size_t o_ht = 0;
};

// The head input and weight are read in 16-byte pieces (their rows then are too: D is a
// multiple of 8).
static bool misaligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) != 0; }

static int32_t check_args(pctc_dtype dtype, int32_t N, const int32_t* T, const int32_t* U, int32_t D, int32_t V,
                          float beam, int32_t chunk) {
  if (dtype != PCTC_F32 && dtype != PCTC_BF16) return PCTC_EINVAL;
  if (N < 0 || D <= 0 || (D % 8) != 0 || D > PCTC_MAX_DIM || V <= 1 || V > PCTC_MAX_VOCAB) return PCTC_EINVAL;
  if (beam != beam) return PCTC_EINVAL;
  if (chunk < 0 || (chunk > 0 && (chunk % 256) != 0)) return PCTC_EINVAL;
  if (N > 0 && (!T || !U)) return PCTC_EINVAL;
  int64_t M = 0, Y = 0;
  for (int n = 0; n < N; ++n) {
    if (T[n] < 1 || U[n] < 0) return PCTC_ELENGTH;
  }
  for (int n = 0; n < N; ++n) {
    if (U[n] > PCTC_MAX_TARGET) return PCTC_ETOOLONG;
    M += T[n];
    Y += U[n];
  }
  if (M > (1LL << 30) || Y > (1LL << 28)) return PCTC_EINVAL;
  return PCTC_OK;
}

// want_dW: the call asks for dW (the union columns' dW_u slices are only needed then).
// allow_e: the layout may serve the two-stream schedule (room for the normaliser's E chunk).
constexpr size_t kEMaxExtra = static_cast<size_t>(64) << 20;
static Layout make_layout(pctc_dtype dtype, int32_t N, const int32_t* T, const int32_t* U, int32_t D, int32_t V,
                          float beam, int32_t chunk, bool want_dW = true, bool allow_e = true) {
  Layout L{};
  L.N = N;
  L.dp = plan_dp(N, T, U, beam);
  L.M = L.dp.M;
  L.Y = L.dp.Y;
  L.pruned = L.dp.pruned;
  L.K_max = (1 + L.Y < V) ? 1 + L.Y : V;
  L.ldS = static_cast<int>(align_up(static_cast<size_t>(L.K_max), 4));
  L.bwd = plan_bwd(dtype == PCTC_BF16 ? 1 : 0, L.M, D, V, chunk);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o += align_up(bytes > 0 ? bytes : 1, 256);
    return at;
  };
  L.o_remap = take(static_cast<size_t>(V) * 4);
  L.o_ubits = take(union_scratch_bytes(V));
  L.o_uids = take(static_cast<size_t>(1 + L.Y) * 4);
  L.o_yrel = take(static_cast<size_t>(L.Y) * 4);
  L.o_small = take(64);
  L.o_status = take(static_cast<size_t>(N) * 4);
  L.o_lossn = take(static_cast<size_t>(N) * 8);
  L.o_lam = take(static_cast<size_t>(L.M) * 8);
  L.o_lam2 = take(static_cast<size_t>(L.M) * 8);
  // bf16: S is dead once the lattice is done; the union columns' [hi | lo] copy of G then uses its room
  size_t s_bytes = static_cast<size_t>(L.M) * L.ldS * 4;
  if (dtype == PCTC_BF16 && union_gb_bytes(L.M, L.K_max) > s_bytes) s_bytes = union_gb_bytes(L.M, L.K_max);
  L.o_S = take(s_bytes);
  L.o_G = take(static_cast<size_t>(L.M) * L.ldS * 4);
  L.o_g = take(static_cast<size_t>(L.M) * 4);
  if (dtype == PCTC_BF16) {  // the overlapped schedule: forecast g and the union-column part
    L.o_gpred = take(static_cast<size_t>(L.M) * 4);
    L.o_pred = take(static_cast<size_t>(N) * 4);
    L.o_corr = take(union_corr_bytes(L.M, D, L.K_max, want_dW));
  }
  L.o_dp = take(L.dp.total);
  L.o_bwd = take(L.bwd.total);
  L.eparts = (dtype == PCTC_BF16 && allow_e) ? lse_e_parts_bf16(L.M, D, V, L.bwd.chunk) : 0;
  const size_t zd_need = static_cast<size_t>(L.M) * L.ldS * sizeof(double);
  const size_t part = lse_partial_bytes(L.M, D);
  size_t e_bytes = 0;  // the first chunk's E rows, written by the normaliser
  if (L.eparts > 0) {
    // the selected logits and the partial pairs then live past the E rows of the gradient
    // buffer; where that tail is too short by more than kEMaxExtra bytes (many frames at a
    // wide head), the first chunk is recomputed instead
    e_bytes = align_up(static_cast<size_t>(L.M) * L.bwd.chunk * 2, 256);
    const size_t tail = L.bwd.dz_bytes > e_bytes ? L.bwd.dz_bytes - e_bytes : 0;
    const size_t lodge = align_up(zd_need, 256) + part;
    if (lodge > tail + kEMaxExtra) {
      L.eparts = 0;
      e_bytes = 0;
    }
  }
  if (L.eparts > 0) {
    e_bytes = align_up(static_cast<size_t>(L.M) * L.bwd.chunk * 2, 256);
    L.o_escale = take(static_cast<size_t>(L.M) * 4);
    L.o_hp = take(static_cast<size_t>(L.M) * D * 2);
    L.o_ht = take(align_up(static_cast<size_t>(D) * L.bwd.Mp * 2, 256));  // H^T [D][Mp] for the normaliser
  }
  // The selected logits in double [M][ldS] (bf16 path) and the normaliser's partial pairs are
  // dead once lambda and S are formed, before the first recompute writes the gradient buffer:
  // they live in that buffer (past the E rows) when it is large enough.
  size_t lent = e_bytes;
  if (dtype == PCTC_BF16) {
    if (L.bwd.dz_bytes >= lent + zd_need) {
      L.o_zd = L.o_bwd + lent;
      lent += align_up(zd_need, 256);
    } else {
      L.o_zd = take(zd_need);
    }
  }
  L.o_part = (L.bwd.dz_bytes >= lent + part) ? L.o_bwd + lent : take(part);
  if (part <= L.bwd.dz_bytes - std::min(L.bwd.dz_bytes, lent)) lent += align_up(part, 256);
  // without E rows the normaliser's H^T also lives in the gradient buffer when it fits there
  // (it is dead before the first recompute), so it costs no memory; otherwise it is not made
  if (dtype == PCTC_BF16 && L.eparts == 0 && L.M > 0 && D % 128 == 0) {
    const size_t ht = align_up(static_cast<size_t>(D) * L.bwd.Mp * 2, 256);
    if (L.bwd.dz_bytes >= lent + ht) L.o_ht = L.o_bwd + lent;
  }
  L.total = o;
  return L;
}

// Host offsets of the utterances: frames, targets, lattice cells.
static void host_offsets(int N, const int32_t* T, const int32_t* U, std::vector<int32_t>& toff,
                         std::vector<int32_t>& yoff, std::vector<int64_t>& soff) {
  toff.assign(N + 1, 0);
  yoff.assign(N + 1, 0);
  soff.assign(N + 1, 0);
  for (int n = 0; n < N; ++n) {
    toff[n + 1] = toff[n] + T[n];
    yoff[n + 1] = yoff[n] + U[n];
    soff[n + 1] = soff[n] + static_cast<int64_t>(T[n]) * (2 * U[n] + 1);
  }
}

// The three offset tables are consecutive in the lattice plan: one copy of a host image of
// that region (img, which must outlive the copy: the callers synchronise before returning).
static hipError_t upload_offsets(const DpPlan& dp, char* dpbase, const std::vector<int32_t>& toff,
                                 const std::vector<int32_t>& yoff, const std::vector<int64_t>& soff,
                                 std::vector<char>& img, hipStream_t stream) {
  img.assign(dp.off_soff + soff.size() * 8 - dp.off_toff, 0);
  memcpy(img.data(), toff.data(), toff.size() * 4);
  memcpy(img.data() + (dp.off_yoff - dp.off_toff), yoff.data(), yoff.size() * 4);
  memcpy(img.data() + (dp.off_soff - dp.off_toff), soff.data(), soff.size() * 8);
  return hipMemcpyAsync(dpbase + dp.off_toff, img.data(), img.size(), hipMemcpyHostToDevice, stream);
}

// Events of the two-stream schedule, reused across calls: a set is taken from a per-device
// pool at the start of a call and returned at its end (after the call has synchronised, so
// every record on it is complete).  Sets are created when the pool is empty and kept until
// the process ends.
constexpr int kCallEvents = 8;
struct CallEvents {
  hipEvent_t e[kCallEvents];
};
static std::mutex g_ev_mu;
static std::map<int, std::vector<CallEvents*>> g_ev_pool;

struct EventsLease {
  int dev = -1;
  CallEvents* set = nullptr;
  hipError_t take() {
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    {
      std::lock_guard<std::mutex> lk(g_ev_mu);
      auto& pool = g_ev_pool[dev];
      if (!pool.empty()) {
        set = pool.back();
        pool.pop_back();
        return hipSuccess;
      }
    }
    CallEvents* c = new CallEvents();
    for (int i = 0; i < kCallEvents; ++i) {
      e = hipEventCreateWithFlags(&c->e[i], hipEventDisableTiming);
      if (e != hipSuccess) {
        for (int j = 0; j < i; ++j) hipEventDestroy(c->e[j]);
        delete c;
        return e;
      }
    }
    set = c;
    return hipSuccess;
  }
  ~EventsLease() {
    if (!set) return;
    std::lock_guard<std::mutex> lk(g_ev_mu);
    g_ev_pool[dev].push_back(set);
  }
};

// Second streams for the lattice stage, which runs beside the dense part of the backward: one
// per caller stream (so that calls on different streams do not queue each other's lattice and
// union work), up to kSideStreams per device, after which caller streams share them by hash.
// Created on first use (default priority, non-blocking) and kept until the process ends.
constexpr int kSideStreams = 4;
static hipError_t side_stream(hipStream_t caller, hipStream_t* out) {
  struct DevSide {
    std::vector<hipStream_t> streams;
    std::map<hipStream_t, hipStream_t> of;
  };
  static std::mutex mu;
  static std::map<int, DevSide> sides;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(mu);
  DevSide& d = sides[dev];
  auto it = d.of.find(caller);
  if (it != d.of.end()) {
    *out = it->second;
    return hipSuccess;
  }
  hipStream_t st = nullptr;
  if (static_cast<int>(d.streams.size()) < kSideStreams) {
    e = hipStreamCreateWithFlags(&st, hipStreamNonBlocking);
    if (e != hipSuccess) return e;
    d.streams.push_back(st);
  } else {
    st = d.streams[std::hash<hipStream_t>{}(caller) % d.streams.size()];
  }
  d.of[caller] = st;
  *out = st;
  return hipSuccess;
}

}  // namespace pctc

using namespace pctc;

extern "C" {

size_t pctc_workspace_size(pctc_dtype dtype, int32_t N, const int32_t* input_lengths, const int32_t* target_lengths,
                           int32_t D, int32_t V, float beam, int32_t chunk) {
  if (check_args(dtype, N, input_lengths, target_lengths, D, V, beam, chunk) != PCTC_OK) return 0;
  return make_layout(dtype, N, input_lengths, target_lengths, D, V, beam, chunk).total;
}

size_t pctc_workspace_size_ex(pctc_dtype dtype, int32_t N, const int32_t* input_lengths,
                              const int32_t* target_lengths, int32_t D, int32_t V, float beam, int32_t chunk,
                              int32_t flags) {
  if (check_args(dtype, N, input_lengths, target_lengths, D, V, beam, chunk) != PCTC_OK) return 0;
  if (flags & ~PCTC_WS_NO_DW) return 0;
  return make_layout(dtype, N, input_lengths, target_lengths, D, V, beam, chunk, !(flags & PCTC_WS_NO_DW)).total;
}

int32_t pctc_normaliser_chunk_columns(pctc_dtype dtype, int32_t N, const int32_t* input_lengths,
                                      const int32_t* target_lengths, int32_t D, int32_t V, float beam,
                                      int32_t chunk, int32_t flags) {
  if (check_args(dtype, N, input_lengths, target_lengths, D, V, beam, chunk) != PCTC_OK) return 0;
  if (flags & ~PCTC_WS_NO_DW) return 0;
  const Layout L = make_layout(dtype, N, input_lengths, target_lengths, D, V, beam, chunk, !(flags & PCTC_WS_NO_DW));
  return L.eparts > 0 ? std::min(L.bwd.chunk, V) : 0;
}

const char* pctc_status_string(int32_t status) {
  switch (status) {
    case PCTC_OK: return "ok";
    case PCTC_EINVAL: return "invalid argument";
    case PCTC_ELABEL: return "target label out of range or equal to blank";
    case PCTC_ELENGTH: return "frame count < 1 or target length < 0";
    case PCTC_EWORKSPACE: return "workspace too small";
    case PCTC_EHIP: return "HIP runtime error";
    case PCTC_ETOOLONG: return "target longer than the supported maximum";
    default: return "unknown status";
  }
}

const char* pctc_last_error(void) { return g_last_error; }

#define PCTC_HIP(call)                         \
  do {                                         \
    hipError_t _e = (call);                    \
    if (_e != hipSuccess) {                    \
      set_error(#call, _e);                    \
      return PCTC_EHIP;                        \
    }                                          \
  } while (0)

int32_t pruned_ctc_fwd_bwd(pctc_dtype dtype, const void* H, int32_t D, const void* W, int32_t V,
                           const int32_t* targets, const int32_t* input_lengths, const int32_t* target_lengths,
                           int32_t N, int32_t blank, float beam, int32_t chunk, double* loss, double* loss_per_utt,
                           int32_t* utt_status, float* dH, float* dW, void* workspace, size_t workspace_bytes,
                           void* stream_ptr) {
  return pruned_ctc_fwd_bwd_ex(dtype, H, D, W, nullptr, V, targets, input_lengths, target_lengths, N, blank, beam,
                               chunk, nullptr, loss, loss_per_utt, utt_status, dH, dW, nullptr, workspace,
                               workspace_bytes, stream_ptr);
}

}  // extern "C"

// The whole path on a workspace laid out by L (arguments checked by the caller).
// two_streams: the bf16 path may run the lattice and the union-column part on a second
// stream beside the dense part of the backward (events are created per call); otherwise
// every step runs on `stream` in Algorithm 1's order.
static int32_t fwd_bwd_run(pctc_dtype dtype, const void* H, int32_t D, const void* W, const float* bias, int32_t V,
                           const int32_t* targets, const int32_t* input_lengths, const int32_t* target_lengths,
                           int32_t N, int32_t blank, float beam, const Layout& L, const float* utt_weight,
                           double* loss, double* loss_per_utt, int32_t* utt_status, float* dH, float* dW, float* db,
                           char* ws, hipStream_t stream, bool two_streams) {
  const int dt = (dtype == PCTC_BF16) ? 1 : 0;
  int32_t* remap = reinterpret_cast<int32_t*>(ws + L.o_remap);
  int32_t* u_ids = reinterpret_cast<int32_t*>(ws + L.o_uids);
  int32_t* y_rel = reinterpret_cast<int32_t*>(ws + L.o_yrel);
  int32_t* Kdev = reinterpret_cast<int32_t*>(ws + L.o_small);
  int32_t* err = Kdev + 1;
  int32_t* status = reinterpret_cast<int32_t*>(ws + L.o_status);
  double* loss_n = reinterpret_cast<double*>(ws + L.o_lossn);
  float2* partials = reinterpret_cast<float2*>(ws + L.o_part);
  double* lam = reinterpret_cast<double*>(ws + L.o_lam);
  float2* lam2 = reinterpret_cast<float2*>(ws + L.o_lam2);
  float* S = reinterpret_cast<float*>(ws + L.o_S);
  float* G = reinterpret_cast<float*>(ws + L.o_G);
  float* g = reinterpret_cast<float*>(ws + L.o_g);
  char* dps = ws + L.o_dp;
  char* bws = ws + L.o_bwd;

  std::vector<int32_t> toff, yoff;
  std::vector<int64_t> soff;
  host_offsets(N, input_lengths, target_lengths, toff, yoff, soff);
  const bool want_bwd = (dH || dW || db);
  int32_t* fflag = Kdev + 2;  // forecast mismatch flag
  const bool overlap = two_streams && (dt == 1) && want_bwd && L.M > 0 && N > 0;
  // the normaliser writes the first chunk's dZ rows as E = exp(z) (dense part only: no bias,
  // no db); einv: its range check, rowscale (escale) and Hp: that chunk's factors
  const bool use_e = overlap && L.eparts > 0 && !bias && !db && (dH || dW);
  // a short lattice (every utterance at most kFrontDeferT frames) starts its front beside the
  // first chunk's dW product, which it slows less than that chunk's dH; a longer one is on the
  // critical path and starts as soon as S is formed
  int t_max = 0;
  for (int n = 0; n < N; ++n) t_max = std::max(t_max, input_lengths[n]);
  const bool defer_front = overlap && t_max <= kFrontDeferT;
  int32_t* einv = Kdev + 3;
  float* escale = use_e ? reinterpret_cast<float*>(ws + L.o_escale) : nullptr;
  ChunkE chunk_e;
  if (use_e) chunk_e = ChunkE{escale, reinterpret_cast<const uint16_t*>(ws + L.o_hp), einv};
  hipStream_t dps_stream = stream;
  struct Events {
    hipEvent_t start = nullptr, sel = nullptr, fork = nullptr, gate0 = nullptr, gate1 = nullptr, dh_done = nullptr,
               join = nullptr, udw = nullptr;
  } ev;
  EventsLease lease;
  std::vector<char> offsets_img;
  float* g_pred = nullptr;
  if (overlap) {
    // Two streams.  Second stream: union/relabel, a forecast of g (-w_n on included
    // utterances) and the masked copy of H it implies, the selected logits (all beside the
    // normaliser pass), later the lattice, the union columns' part of the backward and the
    // final dH reduction.  Caller's stream: the normaliser, S = logits - lambda, and the dense
    // part -g p of the backward beside the lattice.  A wrong forecast (rare: a nonfinite
    // normaliser or a -inf logit on a selected class) is caught and the backward is redone in
    // the plain order.
    PCTC_HIP(side_stream(stream, &dps_stream));
    PCTC_HIP(lease.take());
    ev = Events{lease.set->e[0], lease.set->e[1], lease.set->e[2], lease.set->e[3],
                lease.set->e[4], lease.set->e[5], lease.set->e[6], lease.set->e[7]};
    PCTC_HIP(hipEventRecord(ev.start, stream));
    double* Zd = reinterpret_cast<double*>(ws + L.o_zd);
    // online full-vocabulary log-sum-exp, launched first: it is the longest step (the
    // second stream's wait on the work before it is enqueued after this launch)
    int P = 0;
    if (use_e) {  // also E = exp(z) for the backward's first chunk, into the gradient buffer
      // the frames as H transposed (whole k-lines per copy)
      uint16_t* Ht = L.o_ht ? reinterpret_cast<uint16_t*>(ws + L.o_ht) : nullptr;
      if (Ht)
        PCTC_HIP(launch_ht_build_bf16(static_cast<const uint16_t*>(H), L.M, D, nullptr, nullptr, Ht, L.bwd.Mp, stream));
      PCTC_HIP(launch_lse_partial_e_bf16(static_cast<const uint16_t*>(H), L.M, D, static_cast<const uint16_t*>(W), V,
                                         partials, &P, reinterpret_cast<uint16_t*>(bws), L.bwd.chunk, L.eparts, einv,
                                         stream, Ht, L.bwd.Mp));
    } else if (dt == 1 && !bias && L.o_ht) {
      // no E rows: the same kernel with none of its partitions writing them, frames from H^T
      uint16_t* Ht = reinterpret_cast<uint16_t*>(ws + L.o_ht);
      PCTC_HIP(launch_ht_build_bf16(static_cast<const uint16_t*>(H), L.M, D, nullptr, nullptr, Ht, L.bwd.Mp, stream));
      PCTC_HIP(launch_lse_partial_e_bf16(static_cast<const uint16_t*>(H), L.M, D, static_cast<const uint16_t*>(W), V,
                                         partials, &P, reinterpret_cast<uint16_t*>(bws), L.bwd.chunk, 0, einv, stream,
                                         Ht, L.bwd.Mp));
    } else {
      PCTC_HIP(launch_lse_partials(dt, H, L.M, D, W, bias, V, partials, &P, stream));
    }
    PCTC_HIP(hipStreamWaitEvent(dps_stream, ev.start, 0));
    // beside it: the lattice offsets, Algorithm 1 (union and relabel), the forecast of g and
    // the masked H of the dense part, then the selected logits X W_U^T (+ b_U)
    PCTC_HIP(upload_offsets(L.dp, dps, toff, yoff, soff, offsets_img, dps_stream));
    PCTC_HIP(launch_union_remap(targets, L.Y, blank, V, remap, u_ids, y_rel, Kdev, err, ws + L.o_ubits, dps_stream));
    g_pred = reinterpret_cast<float*>(ws + L.o_gpred);
    int32_t* pred = reinterpret_cast<int32_t*>(ws + L.o_pred);
    PCTC_HIP(launch_g_forecast(L.dp, dps, y_rel, nullptr, utt_weight, g_pred, pred, dps_stream));
    if (dH || dW) {
      uint16_t* Hst = bwd_hst(bws, L.bwd);
      if (Hst)
        PCTC_HIP(launch_ht_build_bf16(static_cast<const uint16_t*>(H), L.M, D, g_pred, bwd_hs(bws, L.bwd), Hst,
                                      L.bwd.Mp, dps_stream));
      else
        PCTC_HIP(launch_hs_build_bf16(static_cast<const uint16_t*>(H), L.M, D, g_pred, bwd_hs(bws, L.bwd), dps_stream));
    }
    PCTC_HIP(launch_gather_s_bf16(static_cast<const uint16_t*>(H), L.M, D, static_cast<const uint16_t*>(W), bias,
                                  u_ids, Kdev, L.K_max, nullptr, nullptr, L.ldS, dps_stream, Zd));
    // the lattice's set-up (zeroing of G and g, per-utterance prep), which does not read S
    PCTC_HIP(launch_ctc_dp(L.dp, input_lengths, target_lengths, S, L.ldS, y_rel, beam, utt_weight, loss_n, status,
                           G, g, nullptr, dps, L.K_max, dps_stream, nullptr, kDpPrep));
    PCTC_HIP(hipEventRecord(ev.sel, dps_stream));
    // S = logits - lambda once both are done
    PCTC_HIP(hipStreamWaitEvent(stream, ev.sel, 0));
    PCTC_HIP(launch_lse_finalize(partials, L.M, P, lam, lam2, Zd, Kdev, S, L.ldS, stream, use_e ? g_pred : nullptr,
                                 escale, einv));
    if (use_e)
      PCTC_HIP(launch_hs_scale_bf16(bwd_hs(bws, L.bwd), L.M, D, einv, escale, reinterpret_cast<uint16_t*>(ws + L.o_hp),
                                    stream));
    if (!defer_front) {
      PCTC_HIP(hipEventRecord(ev.fork, stream));
      PCTC_HIP(hipStreamWaitEvent(dps_stream, ev.fork, 0));
    }
  } else {
    PCTC_HIP(upload_offsets(L.dp, dps, toff, yoff, soff, offsets_img, stream));
    // Algorithm 1: union and relabel
    PCTC_HIP(launch_union_remap(targets, L.Y, blank, V, remap, u_ids, y_rel, Kdev, err, ws + L.o_ubits, stream));
    // online full-vocabulary log-sum-exp, then S = X W_U^T - lambda
    PCTC_HIP(launch_lse(dt, H, L.M, D, W, bias, V, partials, lam, lam2, stream));
    PCTC_HIP(launch_gather_s(dt, H, L.M, D, W, bias, u_ids, Kdev, L.K_max, lam, S, L.ldS, stream));
  }
  // lattice, total scores, zeroing of nonfinite losses, G = dL/dS; then the loss and the
  // per-utterance outputs
  struct DpTail {
    const DpPlan* dp;
    const int32_t *T, *U, *y_rel;
    const float* S;
    int ldS, K_max, N;
    float beam;
    const float* weight;
    double *loss_n, *loss, *loss_per_utt;
    int32_t *status, *utt_status;
    float *G, *g;
    void* dps;
    hipStream_t stream;
    const int32_t* pred;  // forecast to check (two-stream schedule) or null
    int32_t* fflag;
    int phase;
    static hipError_t run(void* p) {
      const DpTail& d = *static_cast<const DpTail*>(p);
      hipError_t e = launch_ctc_dp(*d.dp, d.T, d.U, d.S, d.ldS, d.y_rel, d.beam, d.weight, d.loss_n, d.status, d.G,
                                   d.g, nullptr, d.dps, d.K_max, d.stream, nullptr, d.phase);
      if (e == hipSuccess) e = launch_loss_reduce(d.N, d.loss_n, d.status, d.weight, d.loss, d.stream);
      if (e == hipSuccess && d.loss_per_utt && d.N > 0)
        e = hipMemcpyAsync(d.loss_per_utt, d.loss_n, d.N * sizeof(double), hipMemcpyDeviceToDevice, d.stream);
      if (e == hipSuccess && d.utt_status && d.N > 0)
        e = hipMemcpyAsync(d.utt_status, d.status, d.N * sizeof(int32_t), hipMemcpyDeviceToDevice, d.stream);
      if (e == hipSuccess && d.pred) e = launch_forecast_check(d.N, d.status, d.weight, d.pred, d.fflag, d.stream);
      return e;
    }
  } dpt{&L.dp, input_lengths, target_lengths, y_rel, S, L.ldS, L.K_max, N, beam, utt_weight, loss_n, loss,
        loss_per_utt, status, utt_status, G, g, dps, dps_stream,
        overlap ? reinterpret_cast<const int32_t*>(ws + L.o_pred) : nullptr, fflag, kDpAll};
  if (overlap) {
    // the lattice's front (Viterbi passes and arc mask) now or, deferred, beside the first
    // chunk's dW product; its log-sum passes, occupancies and the loss after the dense part's
    // first chunk, and the union columns' part after its second (see BwdSide)
    DpTail front = dpt;
    front.phase = kDpVit;
    struct FrontWork {
      static hipError_t run(void* p) {
        const DpTail& d = *static_cast<const DpTail*>(p);
        return launch_ctc_dp(*d.dp, d.T, d.U, d.S, d.ldS, d.y_rel, d.beam, d.weight, d.loss_n, d.status, d.G, d.g,
                             nullptr, d.dps, d.K_max, d.stream, nullptr, d.phase);
      }
    };
    if (!defer_front) PCTC_HIP(FrontWork::run(&front));
    dpt.phase = kDpBack;
    // the union columns' part of the backward, from the lattice's G (its frames with g == 0
    // are those of the forecast unless the check fails, and then the backward is redone)
    // With a single split-K slice the dense part accumulates dH in place; the union columns'
    // dH_u is then added once the dense part's last dH product is done (after_dh), instead of
    // being written first and summed in by the final reduction.
    const bool dh_in_place = dH && L.bwd.part_bytes == 0;
    uint16_t* Gb = reinterpret_cast<uint16_t*>(ws + L.o_S);  // S is dead once the lattice is done
    struct UnionWork {
      const float* G;
      int ldG;
      const int32_t *Kdev, *u_ids;
      int K_max, M, D;
      const uint16_t *W, *Hs;
      float* dH;
      bool dh_later, want_dW, want_db;
      void* scratch;
      uint16_t* Gb;
      hipStream_t stream;
      hipEvent_t dw_ready;  // non-null: dW_u is left to the last dense dW launch, which waits for it
      static hipError_t run(void* p) {
        const UnionWork& u = *static_cast<const UnionWork*>(p);
        hipError_t e = launch_union_part_bf16(u.G, u.ldG, u.Kdev, u.K_max, u.u_ids, u.W, u.Hs, u.M, u.D,
                                              u.dh_later ? nullptr : u.dH, u.dh_later, u.want_dW, u.want_db,
                                              u.scratch, u.Gb, u.stream, u.dw_ready != nullptr);
        if (e == hipSuccess && u.dw_ready) e = hipEventRecord(u.dw_ready, u.stream);
        return e;
      }
      static hipError_t run_dh(void* p) {
        const UnionWork& u = *static_cast<const UnionWork*>(p);
        return launch_union_dh_bf16(u.Gb, u.Kdev, u.K_max, u.M, u.D, u.dH, u.scratch, u.want_dW, u.stream);
      }
    } uw{G, L.ldS, Kdev, u_ids, L.K_max, L.M, D, static_cast<const uint16_t*>(W), bwd_hs(bws, L.bwd), dH,
         dh_in_place, dW != nullptr, db != nullptr, ws + L.o_corr, Gb, dps_stream,
         // with dH wanted and at least three chunks the union part is enqueued after the second
         // chunk, well before the last chunk's dW launch, which then also computes dW_u in its
         // last round (with fewer chunks that launch would wait for the whole lattice)
         (dH && dW && L.K_max > 0 && (V + L.bwd.chunk - 1) / L.bwd.chunk >= 3) ? ev.udw : nullptr};
    // dense part, chunk by chunk, on the caller's stream; the final dH reduction, which adds
    // the union part's dH_u (written into dH), runs on the second stream beside the last dW
    BwdSide side;
    side.stream = dps_stream;
    side.gate[0] = ev.gate0;
    side.gate[1] = ev.gate1;
    side.dh_done = ev.dh_done;
    side.reduced = ev.join;
    if (defer_front) {
      side.front = SideWork{&FrontWork::run, &front};
      side.front_gate = ev.fork;
    }
    side.work[0] = SideWork{&DpTail::run, &dpt};
    side.work[1] = SideWork{&UnionWork::run, &uw};
    side.nwork = 2;
    if (dh_in_place) side.after_dh = SideWork{&UnionWork::run_dh, &uw};
    side.dH_extra = (dH && !dh_in_place && L.K_max > 0) ? dH : nullptr;
    side.hs_built = (dH || dW);
    if (use_e) side.ce = &chunk_e;
    if (uw.dw_ready) {
      side.udw = union_dw_extra(L.M, D, L.K_max, Kdev, ws + L.o_corr, Gb);
      side.udw.ready = uw.dw_ready;
    }
    PCTC_HIP(launch_head_bwd(dt, H, L.M, D, W, bias, V, lam2, nullptr, L.ldS, g_pred, nullptr, nullptr, L.ldS, dH, dW,
                             db, bws, L.bwd, stream, &side));
    PCTC_HIP(launch_union_merge_bf16(Kdev, L.K_max, u_ids, L.M, D, dW, db, ws + L.o_corr, stream));
  } else {
    PCTC_HIP(DpTail::run(&dpt));
    // backward: chunk by chunk recomputation
    if (want_bwd)
      PCTC_HIP(launch_head_bwd(dt, H, L.M, D, W, bias, V, lam2, G, L.ldS, g, remap, S, L.ldS, dH, dW, db, bws, L.bwd,
                               stream));
  }
  int32_t hflags[2] = {0, 0};  // label error, forecast mismatch
  PCTC_HIP(hipMemcpyAsync(hflags, err, 2 * sizeof(int32_t), hipMemcpyDeviceToHost, stream));
  PCTC_HIP(hipStreamSynchronize(stream));
  if (overlap && hflags[1] && !hflags[0]) {
    // the union columns' copy of G took the room of S: form S again for the plain-order backward
    PCTC_HIP(launch_gather_s(dt, H, L.M, D, W, bias, u_ids, Kdev, L.K_max, lam, S, L.ldS, stream));
    PCTC_HIP(launch_head_bwd(dt, H, L.M, D, W, bias, V, lam2, G, L.ldS, g, remap, S, L.ldS, dH, dW, db, bws, L.bwd,
                             stream));
    PCTC_HIP(hipStreamSynchronize(stream));
  }
  prof_flush();
  if (hflags[0]) return PCTC_ELABEL;
  return PCTC_OK;
}

// Scratch of the allocation-free entry point: one copy per device, held from the library's
// first use of a device until the process ends.  Host code reaches it only through the
// address hipGetSymbolAddress returns for the current device (noalloc_scratch).
constexpr size_t kNoAllocScratchBytes = static_cast<size_t>(PCTC_NOALLOC_SCRATCH_MIB) << 20;
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

static hipError_t noalloc_scratch(char** out) {
  static std::mutex mu;
  static std::map<int, char*> ptrs;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(mu);
  auto it = ptrs.find(dev);
  if (it == ptrs.end()) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || (reinterpret_cast<uintptr_t>(p) & 255) != 0) return hipErrorInvalidSymbol;
    it = ptrs.emplace(dev, static_cast<char*>(p)).first;
  }
  *out = it->second;
  return hipSuccess;
}

extern "C" {

int32_t pruned_ctc_fwd_bwd_ex(pctc_dtype dtype, const void* H, int32_t D, const void* W, const float* bias, int32_t V,
                              const int32_t* targets, const int32_t* input_lengths, const int32_t* target_lengths,
                              int32_t N, int32_t blank, float beam, int32_t chunk, const float* utt_weight,
                              double* loss, double* loss_per_utt, int32_t* utt_status, float* dH, float* dW,
                              float* db, void* workspace, size_t workspace_bytes, void* stream_ptr) {
  int32_t st = check_args(dtype, N, input_lengths, target_lengths, D, V, beam, chunk);
  if (st != PCTC_OK) return st;
  if (blank < 0 || blank >= V || !loss || !W || misaligned16(W) || misaligned16(H)) return PCTC_EINVAL;
  const Layout L = make_layout(dtype, N, input_lengths, target_lengths, D, V, beam, chunk, dW != nullptr);
  if (L.M > 0 && !H) return PCTC_EINVAL;
  if (L.Y > 0 && !targets) return PCTC_EINVAL;
  if (!workspace || workspace_bytes < L.total) return PCTC_EWORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return PCTC_EINVAL;
  return fwd_bwd_run(dtype, H, D, W, bias, V, targets, input_lengths, target_lengths, N, blank, beam, L, utt_weight,
                     loss, loss_per_utt, utt_status, dH, dW, db, static_cast<char*>(workspace),
                     static_cast<hipStream_t>(stream_ptr), true);
}

size_t pctc_noalloc_scratch_bytes(void) { return kNoAllocScratchBytes; }

int32_t pruned_ctc_fwd_bwd_noalloc(pctc_dtype dtype, const void* H, int32_t D, const void* W, const float* bias,
                                   int32_t V, const int32_t* targets, const int32_t* input_lengths,
                                   const int32_t* target_lengths, int32_t N, int32_t blank, float beam, int32_t chunk,
                                   const float* utt_weight, double* loss, double* loss_per_utt, int32_t* utt_status,
                                   float* dH, float* dW, float* db, void* stream_ptr) {
  int32_t st = check_args(dtype, N, input_lengths, target_lengths, D, V, beam, chunk);
  if (st != PCTC_OK) return st;
  if (blank < 0 || blank >= V || !loss || !W || misaligned16(W) || misaligned16(H)) return PCTC_EINVAL;
  Layout L = make_layout(dtype, N, input_lengths, target_lengths, D, V, beam, chunk, dW != nullptr, false);
  if (chunk == 0 && L.total > kNoAllocScratchBytes) {
    // the widest backward chunk (a multiple of 256 columns) whose layout fits the scratch;
    // the layout is not monotone in the chunk (the dH product's split count changes with
    // it), so every width is tried from the default down
    for (int c = L.bwd.chunk / 256 * 256; c >= 256; c -= 256) {
      const Layout Lc = make_layout(dtype, N, input_lengths, target_lengths, D, V, beam, c, dW != nullptr, false);
      if (Lc.total <= kNoAllocScratchBytes) {
        L = Lc;
        break;
      }
    }
  }
  if (L.total > kNoAllocScratchBytes) {
    snprintf(g_last_error, sizeof(g_last_error),
             "the batch needs %zu bytes of scratch; the allocation-free entry point holds %zu", L.total,
             kNoAllocScratchBytes);
    return PCTC_EWORKSPACE;
  }
  if (L.M > 0 && !H) return PCTC_EINVAL;
  if (L.Y > 0 && !targets) return PCTC_EINVAL;
  char* ws = nullptr;
  PCTC_HIP(noalloc_scratch(&ws));
  return fwd_bwd_run(dtype, H, D, W, bias, V, targets, input_lengths, target_lengths, N, blank, beam, L, utt_weight,
                     loss, loss_per_utt, utt_status, dH, dW, db, ws, static_cast<hipStream_t>(stream_ptr), false);
}

size_t pctc_union_scratch_bytes(int32_t V) { return (V <= 1 || V > PCTC_MAX_VOCAB) ? 0 : union_scratch_bytes(V); }

int32_t pctc_union_remap(const int32_t* targets, int32_t total_targets, int32_t blank, int32_t V, int32_t* remap,
                         int32_t* u_ids, int32_t* y_rel, int32_t* K, int32_t* err, void* scratch, void* stream_ptr) {
  if (V <= 1 || V > PCTC_MAX_VOCAB || blank < 0 || blank >= V || total_targets < 0) return PCTC_EINVAL;
  if (!remap || !u_ids || !K || !err || !scratch || (total_targets > 0 && (!targets || !y_rel))) return PCTC_EINVAL;
  hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
  PCTC_HIP(launch_union_remap(targets, total_targets, blank, V, remap, u_ids, y_rel, K, err, scratch, stream));
  int32_t herr = 0;
  PCTC_HIP(hipMemcpyAsync(&herr, err, sizeof(int32_t), hipMemcpyDeviceToHost, stream));
  PCTC_HIP(hipStreamSynchronize(stream));
  prof_flush();
  return herr ? PCTC_ELABEL : PCTC_OK;
}

size_t pctc_lse_scratch_bytes(int32_t M, int32_t D) {
  return (M < 0 || D <= 0 || D > PCTC_MAX_DIM) ? 0
                           : lse_partial_bytes(M, D) + align_up(static_cast<size_t>(M > 0 ? M : 1) * sizeof(float2), 256);
}

int32_t pctc_lse_select(pctc_dtype dtype, const void* H, int32_t M, int32_t D, const void* W, int32_t V,
                        const int32_t* u_ids, const int32_t* K, int32_t K_max, double* lam, float* S, int32_t ldS,
                        void* partials, void* stream_ptr) {
  if ((dtype != PCTC_F32 && dtype != PCTC_BF16) || M < 0 || D <= 0 || D % 8 || D > PCTC_MAX_DIM || V <= 1 || K_max < 1 ||
      ldS < K_max || !W || !lam || !partials || (M > 0 && !H) || misaligned16(W) || misaligned16(H))
    return PCTC_EINVAL;
  hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
  const int dt = (dtype == PCTC_BF16) ? 1 : 0;
  // scratch = [partials][lam2]
  float2* lam2 = reinterpret_cast<float2*>(static_cast<char*>(partials) + lse_partial_bytes(M, D));
  PCTC_HIP(launch_lse(dt, H, M, D, W, nullptr, V, static_cast<float2*>(partials), lam, lam2, stream));
  if (S && u_ids && K) PCTC_HIP(launch_gather_s(dt, H, M, D, W, nullptr, u_ids, K, K_max, lam, S, ldS, stream));
  PCTC_HIP(hipStreamSynchronize(stream));
  prof_flush();
  return PCTC_OK;
}

size_t pctc_dp_scratch_bytes(int32_t N, const int32_t* input_lengths, const int32_t* target_lengths, float beam) {
  if (N < 0 || (N > 0 && (!input_lengths || !target_lengths))) return 0;
  for (int n = 0; n < N; ++n)
    if (input_lengths[n] < 1 || target_lengths[n] < 0 || target_lengths[n] > PCTC_MAX_TARGET) return 0;
  return plan_dp(N, input_lengths, target_lengths, beam).total;
}

int32_t pctc_ctc_dp(const float* S, int32_t ldS, int32_t K_max, const int32_t* y_rel, const int32_t* input_lengths,
                    const int32_t* target_lengths, int32_t N, float beam, double* loss_per_utt, int32_t* utt_status,
                    float* G, float* g, uint8_t* keep_mask, void* dp_scratch, void* stream_ptr) {
  if (N < 0 || beam != beam || ldS < K_max || K_max < 1) return PCTC_EINVAL;
  if (N > 0 && (!input_lengths || !target_lengths || !loss_per_utt || !utt_status || !dp_scratch)) return PCTC_EINVAL;
  for (int n = 0; n < N; ++n) {
    if (input_lengths[n] < 1 || target_lengths[n] < 0) return PCTC_ELENGTH;
    if (target_lengths[n] > PCTC_MAX_TARGET) return PCTC_ETOOLONG;
  }
  hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
  const DpPlan dp = plan_dp(N, input_lengths, target_lengths, beam);
  if (dp.M > 0 && (!S || !G || !g)) return PCTC_EINVAL;
  std::vector<int32_t> toff, yoff;
  std::vector<int64_t> soff;
  host_offsets(N, input_lengths, target_lengths, toff, yoff, soff);
  char* dps = static_cast<char*>(dp_scratch);
  std::vector<char> img;
  PCTC_HIP(upload_offsets(dp, dps, toff, yoff, soff, img, stream));
  PCTC_HIP(launch_ctc_dp(dp, input_lengths, target_lengths, S, ldS, y_rel, beam, nullptr, loss_per_utt, utt_status, G, g,
                         keep_mask, dps, K_max, stream, nullptr));
  PCTC_HIP(hipStreamSynchronize(stream));
  prof_flush();
  return PCTC_OK;
}

// Greedy decode workspace: argmax partials, frame offsets, and the ids when not returned.
static size_t greedy_layout(int32_t N, int32_t M, int32_t D, size_t* o_toff, size_t* o_ids) {
  const size_t part = lse_partial_bytes(M > 0 ? M : 1, D);
  *o_toff = part;
  *o_ids = part + align_up(static_cast<size_t>(N + 1) * sizeof(int32_t), 256);
  return *o_ids + align_up(static_cast<size_t>(M > 0 ? M : 1) * sizeof(int32_t), 256);
}

size_t pctc_greedy_workspace_size(int32_t N, int32_t M, int32_t D) {
  if (N < 0 || M < 0 || D <= 0 || D > PCTC_MAX_DIM) return 0;
  size_t a, b;
  return greedy_layout(N, M, D, &a, &b);
}

int32_t pctc_greedy_decode(pctc_dtype dtype, const void* H, int32_t D, const void* W, const float* bias, int32_t V,
                           const int32_t* input_lengths, int32_t N, int32_t blank, int32_t* ids, int32_t* tokens,
                           int32_t* token_lengths, void* workspace, size_t workspace_bytes, void* stream_ptr) {
  if ((dtype != PCTC_F32 && dtype != PCTC_BF16) || N < 0 || D <= 0 || D % 8 || D > PCTC_MAX_DIM || V <= 1 || V > PCTC_MAX_VOCAB ||
      blank < 0 || blank >= V || !W || misaligned16(W) || misaligned16(H))
    return PCTC_EINVAL;
  if (N > 0 && !input_lengths) return PCTC_EINVAL;
  int64_t M64 = 0;
  for (int n = 0; n < N; ++n) {
    if (input_lengths[n] < 1) return PCTC_ELENGTH;
    M64 += input_lengths[n];
  }
  if (M64 > INT32_MAX) return PCTC_EINVAL;
  const int M = static_cast<int>(M64);
  if (M > 0 && (!H || !tokens || !token_lengths)) return PCTC_EINVAL;
  size_t o_toff, o_ids;
  const size_t need = greedy_layout(N, M, D, &o_toff, &o_ids);
  if (!workspace || workspace_bytes < need) return PCTC_EWORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return PCTC_EINVAL;
  if (N == 0) return PCTC_OK;
  hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
  char* ws = static_cast<char*>(workspace);
  std::vector<int32_t> toff(N + 1, 0);
  for (int n = 0; n < N; ++n) toff[n + 1] = toff[n] + input_lengths[n];
  int32_t* dtoff = reinterpret_cast<int32_t*>(ws + o_toff);
  PCTC_HIP(hipMemcpyAsync(dtoff, toff.data(), (N + 1) * sizeof(int32_t), hipMemcpyHostToDevice, stream));
  int32_t* idv = ids ? ids : reinterpret_cast<int32_t*>(ws + o_ids);
  PCTC_HIP(launch_greedy(dtype == PCTC_BF16 ? 1 : 0, H, M, D, W, bias, V, dtoff, N, blank,
                         reinterpret_cast<float2*>(ws), idv, tokens, token_lengths, stream));
  PCTC_HIP(hipStreamSynchronize(stream));  // the host offsets must outlive the copy
  prof_flush();
  return PCTC_OK;
}

size_t pctc_discarded_mass_scratch_bytes(int32_t N, const int32_t* input_lengths, const int32_t* target_lengths) {
  if (N < 0 || (N > 0 && (!input_lengths || !target_lengths))) return 0;
  for (int n = 0; n < N; ++n)
    if (input_lengths[n] < 1 || target_lengths[n] < 0 || target_lengths[n] > PCTC_MAX_TARGET) return 0;
  return plan_dp(N, input_lengths, target_lengths, 1.f).total;
}

int32_t pctc_discarded_mass(const float* S, int32_t ldS, int32_t K_max, const int32_t* y_rel,
                            const int32_t* input_lengths, const int32_t* target_lengths, int32_t N, const float* beams,
                            int32_t nbeams, double* delta, void* dp_scratch, void* stream_ptr) {
  if (N < 0 || nbeams < 0 || ldS < K_max || K_max < 1 || (nbeams > 0 && !beams)) return PCTC_EINVAL;
  for (int b = 0; b < nbeams; ++b)
    if (!(beams[b] >= 0.f) || !(beams[b] < INFINITY)) return PCTC_EINVAL;  // finite, non-negative
  for (int n = 0; n < N; ++n) {
    if (input_lengths[n] < 1 || target_lengths[n] < 0) return PCTC_ELENGTH;
    if (target_lengths[n] > PCTC_MAX_TARGET) return PCTC_ETOOLONG;
  }
  if (N == 0 || nbeams == 0) return PCTC_OK;
  if (!S || !delta || !dp_scratch) return PCTC_EINVAL;
  hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
  const DpPlan dp = plan_dp(N, input_lengths, target_lengths, 1.f);
  std::vector<int32_t> toff, yoff;
  std::vector<int64_t> soff;
  host_offsets(N, input_lengths, target_lengths, toff, yoff, soff);
  std::vector<char> img;
  PCTC_HIP(upload_offsets(dp, static_cast<char*>(dp_scratch), toff, yoff, soff, img, stream));
  PCTC_HIP(launch_discarded_mass(dp, S, ldS, y_rel, beams, nbeams, delta, dp_scratch, K_max, stream));
  PCTC_HIP(hipStreamSynchronize(stream));
  prof_flush();
  return PCTC_OK;
}

// Stage entry scratch: the backward plan, then u_ids [ldG], K, and S [M][ldG].
struct BwdStageLayout {
  BwdPlan plan;
  size_t o_uids, o_K, o_S, total;
};
static BwdStageLayout bwd_stage_layout(int dt, int M, int D, int V, int ldG, int chunk) {
  BwdStageLayout b;
  b.plan = plan_bwd(dt, M, D, V, chunk);
  b.o_uids = b.plan.total;
  b.o_K = b.o_uids + align_up(static_cast<size_t>(ldG) * 4, 256);
  b.o_S = b.o_K + 256;
  b.total = b.o_S + align_up(static_cast<size_t>(M) * ldG * 4, 256);
  return b;
}

size_t pctc_bwd_scratch_bytes(pctc_dtype dtype, int32_t M, int32_t D, int32_t V, int32_t ldG, int32_t chunk) {
  if ((dtype != PCTC_F32 && dtype != PCTC_BF16) || M < 0 || D <= 0 || D > PCTC_MAX_DIM || V <= 1 || ldG < 1 || chunk < 0 ||
      (chunk > 0 && chunk % 256))
    return 0;
  return bwd_stage_layout(dtype == PCTC_BF16 ? 1 : 0, M, D, V, ldG, chunk).total;
}

int32_t pctc_bwd_chunk(pctc_dtype dtype, int32_t M, int32_t D, int32_t V, int32_t chunk) {
  if ((dtype != PCTC_F32 && dtype != PCTC_BF16) || M < 0 || D <= 0 || D > PCTC_MAX_DIM || V <= 1 || chunk < 0 ||
      (chunk > 0 && chunk % 256))
    return 0;
  return plan_bwd(dtype == PCTC_BF16 ? 1 : 0, M, D, V, chunk).chunk;
}

int32_t pctc_head_bwd(pctc_dtype dtype, const void* H, int32_t M, int32_t D, const void* W, int32_t V,
                      const double* lam, const float* G, int32_t ldG, const float* g, const int32_t* remap,
                      int32_t chunk, float* dH, float* dW, void* bwd_scratch, void* stream_ptr) {
  if ((dtype != PCTC_F32 && dtype != PCTC_BF16) || M < 0 || D <= 0 || D % 8 || D > PCTC_MAX_DIM || V <= 1 || chunk < 0 ||
      (chunk > 0 && chunk % 256) || !W || !bwd_scratch || ldG < 1 || misaligned16(W) || misaligned16(H))
    return PCTC_EINVAL;
  if (M > 0 && (!H || !lam || !G || !g || !remap)) return PCTC_EINVAL;
  hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
  const int dt = (dtype == PCTC_BF16) ? 1 : 0;
  const BwdStageLayout b = bwd_stage_layout(dt, M, D, V, ldG, chunk);
  const BwdPlan& plan = b.plan;
  char* sc = static_cast<char*>(bwd_scratch);
  float2* lam2 = reinterpret_cast<float2*>(sc + plan.dz_bytes + plan.ht_bytes + plan.part_bytes);
  int32_t* u_ids = reinterpret_cast<int32_t*>(sc + b.o_uids);
  int32_t* Kdev = reinterpret_cast<int32_t*>(sc + b.o_K);
  float* S = reinterpret_cast<float*>(sc + b.o_S);
  PCTC_HIP(launch_lam2(lam, M, lam2, stream));
  if (dt == 1 && M > 0) {
    // the union and its selected log-probabilities, as the forward would have left them
    PCTC_HIP(launch_remap_invert(remap, V, u_ids, Kdev, stream));
    PCTC_HIP(launch_gather_s(dt, H, M, D, W, nullptr, u_ids, Kdev, ldG, lam, S, ldG, stream));
  }
  PCTC_HIP(launch_head_bwd(dt, H, M, D, W, nullptr, V, lam2, G, ldG, g, remap, S, ldG, dH, dW, nullptr, bwd_scratch,
                           plan, stream));
  PCTC_HIP(hipStreamSynchronize(stream));
  prof_flush();
  return PCTC_OK;
}

// Grouped logits: one workspace serves both directions.
//   [small 256 B][remap V][ forward: partials | lse_O | lam2 | zero | complement bias ]
//                         [ backward: G M x K | g | lam2 | recomputed-backward scratch ]
struct GroupedLayout {
  BwdPlan plan;
  size_t o_remap, o_part, o_lamo, o_lam2f, o_zero, o_bo, o_G, o_g, o_lam2b, o_bwd, total;
};
static GroupedLayout grouped_layout(int dt, int M, int D, int V, int K, int chunk) {
  GroupedLayout L;
  const size_t m8 = align_up(static_cast<size_t>(M > 0 ? M : 1) * 8, 256);
  L.plan = plan_bwd(dt, M, D, V, chunk);
  L.o_remap = 256;
  L.o_part = L.o_remap + align_up(static_cast<size_t>(V) * 4, 256);
  L.o_lamo = L.o_part + lse_partial_bytes(M, D);
  L.o_lam2f = L.o_lamo + m8;
  L.o_zero = L.o_lam2f + m8;
  L.o_bo = L.o_zero + m8;
  const size_t fwd_end = L.o_bo + align_up(static_cast<size_t>(V) * 4, 256);
  L.o_G = L.o_part;
  L.o_g = L.o_G + align_up(static_cast<size_t>(M) * K * 4, 256);
  L.o_lam2b = L.o_g + align_up(static_cast<size_t>(M > 0 ? M : 1) * 4, 256);
  L.o_bwd = L.o_lam2b + m8;
  const size_t bwd_end = L.o_bwd + L.plan.total;
  L.total = fwd_end > bwd_end ? fwd_end : bwd_end;
  return L;
}

static bool grouped_args_ok(pctc_dtype dtype, int32_t M, int32_t D, int32_t V, int32_t K, int32_t chunk) {
  return (dtype == PCTC_F32 || dtype == PCTC_BF16) && M >= 0 && D > 0 && D % 8 == 0 && D <= PCTC_MAX_DIM && V > 1 && K >= 1 && K <= V &&
         chunk >= 0 && (chunk == 0 || chunk % 256 == 0) && static_cast<int64_t>(M) * (K + 1) <= INT32_MAX;
}

// Builds remap from u_ids and reads the error flag back (synchronous).
static int32_t grouped_index(const int32_t* u_ids, int32_t K, int32_t V, char* ws, hipStream_t stream) {
  int32_t* small = reinterpret_cast<int32_t*>(ws);
  int32_t* remap = reinterpret_cast<int32_t*>(ws + 256);
  PCTC_HIP(launch_grouped_index(u_ids, K, V, remap, small, stream));
  int32_t herr = 0;
  PCTC_HIP(hipMemcpyAsync(&herr, small + 1, sizeof(int32_t), hipMemcpyDeviceToHost, stream));
  PCTC_HIP(hipStreamSynchronize(stream));
  return herr ? PCTC_ELABEL : PCTC_OK;
}

size_t pctc_grouped_workspace_size(pctc_dtype dtype, int32_t M, int32_t D, int32_t V, int32_t K, int32_t chunk) {
  if (!grouped_args_ok(dtype, M, D, V, K, chunk)) return 0;
  return grouped_layout(dtype == PCTC_BF16 ? 1 : 0, M, D, V, K, chunk).total;
}

int32_t pctc_grouped_logprobs(pctc_dtype dtype, const void* H, int32_t M, int32_t D, const void* W, const float* bias,
                              int32_t V, const int32_t* u_ids, int32_t K, float* logp, double* lam, void* workspace,
                              size_t workspace_bytes, void* stream_ptr) {
  if (!grouped_args_ok(dtype, M, D, V, K, 0) || !W || !u_ids || misaligned16(W) || misaligned16(H)) return PCTC_EINVAL;
  if (M > 0 && (!H || !logp || !lam)) return PCTC_EINVAL;
  const int dt = (dtype == PCTC_BF16) ? 1 : 0;
  const GroupedLayout L = grouped_layout(dt, M, D, V, K, 0);
  if (!workspace || workspace_bytes < L.total) return PCTC_EWORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return PCTC_EINVAL;
  hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
  char* ws = static_cast<char*>(workspace);
  const int32_t st = grouped_index(u_ids, K, V, ws, stream);
  if (st != PCTC_OK || M == 0) return st;
  const int32_t* Kdev = reinterpret_cast<const int32_t*>(ws);
  const int32_t* remap = reinterpret_cast<const int32_t*>(ws + L.o_remap);
  double* lse_o = reinterpret_cast<double*>(ws + L.o_lamo);
  double* zero = reinterpret_cast<double*>(ws + L.o_zero);
  float* bo = reinterpret_cast<float*>(ws + L.o_bo);
  if (K < V) {
    // the complement's log-sum-exp: the normaliser pass with the selected rows masked out
    PCTC_HIP(launch_grouped_comp_bias(bias, remap, V, bo, stream));
    PCTC_HIP(launch_lse(dt, H, M, D, W, bo, V, reinterpret_cast<float2*>(ws + L.o_part), lse_o,
                        reinterpret_cast<float2*>(ws + L.o_lam2f), stream));
  } else {
    PCTC_HIP(launch_fill_d(lse_o, M, -INFINITY, stream));
  }
  // raw selected logits into the first K columns of each exported row
  PCTC_HIP(launch_fill_d(zero, M, 0.0, stream));
  PCTC_HIP(launch_gather_s(dt, H, M, D, W, bias, u_ids, Kdev, K, zero, logp, K + 1, stream));
  PCTC_HIP(launch_grouped_finalize(logp, K, M, lse_o, lam, stream));
  PCTC_HIP(hipStreamSynchronize(stream));
  prof_flush();
  return PCTC_OK;
}

int32_t pctc_grouped_backward(pctc_dtype dtype, const void* H, int32_t M, int32_t D, const void* W, const float* bias,
                              int32_t V, const int32_t* u_ids, int32_t K, const float* logp, const double* lam,
                              const float* dlogp, int32_t chunk, float* dH, float* dW, float* db, void* workspace,
                              size_t workspace_bytes, void* stream_ptr) {
  if (!grouped_args_ok(dtype, M, D, V, K, chunk) || !W || !u_ids || misaligned16(W) || misaligned16(H))
    return PCTC_EINVAL;
  if (M > 0 && (!H || !logp || !lam || !dlogp)) return PCTC_EINVAL;
  const int dt = (dtype == PCTC_BF16) ? 1 : 0;
  const GroupedLayout L = grouped_layout(dt, M, D, V, K, chunk);
  if (!workspace || workspace_bytes < L.total) return PCTC_EWORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255) != 0) return PCTC_EINVAL;
  hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
  char* ws = static_cast<char*>(workspace);
  const int32_t st = grouped_index(u_ids, K, V, ws, stream);
  if (st != PCTC_OK) return st;
  if (!dH && !dW && !db) return PCTC_OK;
  const int32_t* remap = reinterpret_cast<const int32_t*>(ws + L.o_remap);
  float* G = reinterpret_cast<float*>(ws + L.o_G);
  float* g = reinterpret_cast<float*>(ws + L.o_g);
  float2* lam2 = reinterpret_cast<float2*>(ws + L.o_lam2b);
  PCTC_HIP(launch_grouped_adapter(logp, dlogp, K, M, G, g, stream));
  PCTC_HIP(launch_lam2(lam, M, lam2, stream));
  PCTC_HIP(launch_head_bwd(dt, H, M, D, W, bias, V, lam2, G, K, g, remap, logp, K + 1, dH, dW, db, ws + L.o_bwd,
                           L.plan, stream));
  PCTC_HIP(hipStreamSynchronize(stream));
  prof_flush();
  return PCTC_OK;
}

void pctc_prof_enable(int32_t on) { prof_state().enabled = (on != 0); }

void pctc_prof_select(const char* name) {
  ProfState& s = prof_state();
  std::lock_guard<std::mutex> lk(s.mu);
  s.only = name ? name : "";
}

void pctc_prof_reset(void) {
  ProfState& s = prof_state();
  std::lock_guard<std::mutex> lk(s.mu);
  prof_resolve(s);  // recycles the pending pairs; their times belong to the cleared totals
  s.totals.clear();
  s.names.clear();
}

int32_t pctc_prof_count(void) {
  ProfState& s = prof_state();
  std::lock_guard<std::mutex> lk(s.mu);
  prof_resolve(s);
  return static_cast<int32_t>(s.names.size());
}

int32_t pctc_prof_get(int32_t i, const char** name, double* total_ms, int64_t* launches) {
  ProfState& s = prof_state();
  std::lock_guard<std::mutex> lk(s.mu);
  prof_resolve(s);
  if (i < 0 || i >= static_cast<int32_t>(s.names.size())) return 0;
  const auto& t = s.totals[s.names[i]];
  if (name) *name = s.names[i].c_str();
  if (total_ms) *total_ms = t.first;
  if (launches) *launches = t.second;
  return 1;
}

}  // extern "C"
