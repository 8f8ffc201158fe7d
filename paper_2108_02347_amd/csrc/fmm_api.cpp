// C ABI of the FMMformer attention forward operator: argument validation,
// segment planning, the per-(device, stream) workspace cache and the optional
// kernel timer.  Every kernel is launched asynchronously on the caller's stream.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#include <algorithm>
#include <atomic>
#include <map>
#include <mutex>
#include <random>
#include <utility>
#include <vector>

#include "../../include/fmm_attn.h"
#include "fmm_launch.h"
#include "fmm_fw.h"

namespace {

constexpr int kVersion = 1 * 10000 + 2 * 100 + 0;

// ------------------------------------------------------------------ planning
// Segments split the key axis of every (batch, head) slice for the far-field
// state: enough segments to give the GPU about 512 workgroups, but long enough
// that the per-segment state (rank * d * (d+1) floats) stays at most a quarter
// of the key/value bytes it summarises.
struct Plan {
  int nseg;
  int L;
  int nseg_apply;
  int L_apply;
  size_t ws_bytes;
  int fused_g = 0;  // workgroups per slice of the one-launch path (0: not available)
};

// The one-launch path for short non-causal slices is planned for MI355X's 256
// compute units at two workgroups each; a device with fewer CUs (checked per
// call) takes the three-launch path with the same workspace.
constexpr int kFusedPlanWorkgroups = 512;

// Rows per segment so that B*H*segments is about `target_wg` workgroups.
long long seg_rows(long long bh, int N, long long target_wg, int tm) {
  const long long per_slice = bh >= target_wg ? 1 : (target_wg + bh - 1) / bh;
  long long L = (N + per_slice - 1) / per_slice;
  L = (L + tm - 1) / tm * tm;
  return L < tm ? tm : L;
}

Plan make_plan(int B, int H, int N, int d, int rank, int esize, int apply_tm) {
  const int tm = fmm::tile_rows();
  const long long bh = (long long)B * H;
  // state segments: ~512 workgroups, but each segment's state record
  // (rank*d*(d+1) floats) at most a quarter of the K+V bytes it summarises
  long long L = seg_rows(bh, N, 512, tm);
  const long long lmin = 8LL * rank * (d + 1) / esize;
  if (L < lmin) L = (lmin + tm - 1) / tm * tm;
  // non-causal apply walk: ~512 workgroups (two per CU), no state per segment
  const long long La = seg_rows(bh, N, 512, apply_tm);
  Plan p;
  p.L = (int)L;
  p.nseg = (int)((N + L - 1) / L);
  p.L_apply = (int)La;
  p.nseg_apply = (int)((N + La - 1) / La);
  typedef unsigned __int128 u128;
  const u128 rec = (u128)rank * d * (d + 1);
  const u128 ws = ((u128)bh * p.nseg + (u128)bh) * rec * sizeof(float);
  // a workspace beyond half the address space cannot exist: report it as 0
  p.ws_bytes = ws > (u128)(SIZE_MAX / 2) ? 0 : (size_t)((ws + 255) / 256 * 256);
  return p;
}

bool supported(int d, int rank) {
  return (d == 16 || d == 32 || d == 64 || d == 128) && rank >= 1 && rank <= 3;
}

bool overlaps(const void* a, const void* b, size_t n) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + n && y < x + n;
}
// [a, a + na) and [b, b + nb) share a byte
bool overlaps2(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}

int validate(const void* q, const void* k, const void* v, void* out, int B, int H, int N,
             int d, int band_k, int rank, int causal, const float* w_near, const float* w_far,
             int dtype, int far_norm) {
  if (!q || !k || !v || !out || !w_near || !w_far) return FMM_ERR_INVALID_ARG;
  if (B < 1 || H < 1 || N < 1 || d < 1 || band_k < 0) return FMM_ERR_INVALID_ARG;
  if (causal != 0 && causal != 1) return FMM_ERR_INVALID_ARG;
  if (far_norm != FMM_FAR_NORM_PER_MAP && far_norm != FMM_FAR_NORM_JOINT)
    return FMM_ERR_INVALID_ARG;
  if (dtype != FMM_DTYPE_F32 && dtype != FMM_DTYPE_BF16) return FMM_ERR_UNSUPPORTED;
  if (!supported(d, rank)) return FMM_ERR_UNSUPPORTED;
  const size_t es = dtype == FMM_DTYPE_BF16 ? 2 : 4;
  // sizes in 128-bit arithmetic: four positive ints cannot overflow it
  typedef unsigned __int128 u128;
  const u128 bytes128 = (u128)(unsigned)B * (unsigned)H * (unsigned)N * (unsigned)d * es;
  if (bytes128 > (u128)INT64_MAX) return FMM_ERR_INVALID_ARG;
  // slices are counted in int by the launchers; grids are checked before launch
  if ((long long)B * H > INT32_MAX) return FMM_ERR_UNSUPPORTED;
  for (const void* p : {q, k, v, (const void*)out})
    if ((uintptr_t)p % 16) return FMM_ERR_INVALID_ARG;
  if ((uintptr_t)w_near % 4 || (uintptr_t)w_far % 4) return FMM_ERR_INVALID_ARG;
  const size_t bytes = (size_t)bytes128;
  if (overlaps(out, q, bytes) || overlaps(out, k, bytes) || overlaps(out, v, bytes))
    return FMM_ERR_INVALID_ARG;
  return FMM_OK;
}

// ------------------------------------------------------------------ timing
struct EventTimer : fmm::LaunchTimer {
  std::mutex mu;
  bool enabled = false;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pending[FMM_KERNEL_COUNT];
  std::vector<hipEvent_t> pool;

  hipEvent_t take_one() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
  bool take(int, hipEvent_t* start, hipEvent_t* stop) override {
    if (!enabled) return false;
    *start = take_one();
    *stop = take_one();
    if (*start && *stop) return true;
    if (*start) pool.push_back(*start);
    if (*stop) pool.push_back(*stop);
    return false;
  }
  void commit(int kernel, hipEvent_t start, hipEvent_t stop) override {
    pending[kernel].push_back({start, stop});
  }
};

EventTimer& timer() {
  static EventTimer* t = new EventTimer();
  return *t;
}

// ------------------------------------------------------------------ workspace
struct WsEntry {
  void* ptr = nullptr;
  size_t bytes = 0;
};

std::mutex& ws_mutex() {
  static std::mutex* m = new std::mutex();
  return *m;
}
std::map<std::pair<int, void*>, WsEntry>& ws_map() {
  static auto* m = new std::map<std::pair<int, void*>, WsEntry>();
  return *m;
}

size_t ws_limit() {
  const char* s = getenv("FMM_ATTN_WS_LIMIT");
  if (!s || !*s) return (size_t)-1;
  return (size_t)strtoull(s, nullptr, 10);
}

// Returns a workspace of at least `bytes` for (current device, stream).  The
// caller holds ws_mutex() until its kernels are enqueued, so no other thread
// can free the buffer between this lookup and the launches that use it.
int acquire_ws_locked(void* stream, size_t bytes, void** out) {
  if (bytes > ws_limit()) return FMM_ERR_OOM;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return FMM_ERR_HIP;
  WsEntry& e = ws_map()[{dev, stream}];
  if (e.bytes < bytes) {
    // a stream under graph capture can neither allocate nor synchronise: its
    // workspace has to come from an earlier call outside the capture
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing((hipStream_t)stream, &cs) != hipSuccess) {
      (void)hipGetLastError();
      return FMM_ERR_HIP;
    }
    if (cs != hipStreamCaptureStatusNone) return FMM_ERR_UNSUPPORTED;
    if (e.ptr) {
      // kernels enqueued earlier on this stream may still read the old buffer
      if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return FMM_ERR_HIP;
      (void)hipFree(e.ptr);
      e.ptr = nullptr;
      e.bytes = 0;
    }
    void* p = nullptr;
    if (hipMalloc(&p, bytes) != hipSuccess) {
      (void)hipGetLastError();
      return FMM_ERR_OOM;
    }
    e.ptr = p;
    e.bytes = bytes;
  }
  *out = e.ptr;
  return FMM_OK;
}

// The dry pass over the launch sequence: grid limits and LDS limits, nothing
// enqueued.  Runs before any workspace is acquired.
int check_launch(const fmm::LaunchArgs& a) {
  EventTimer& t = timer();
  std::lock_guard<std::mutex> g(t.mu);
  fmm::Launcher dry;
  dry.timer = &t;
  dry.dry = true;
  if (fmm::launch_forward(a, dry) != hipSuccess)
    return dry.err == hipErrorInvalidConfiguration ? FMM_ERR_UNSUPPORTED : FMM_ERR_HIP;
  return FMM_OK;
}

// Enqueues the launch sequence (after check_launch passed).
int launch_now(const fmm::LaunchArgs& a) {
  EventTimer& t = timer();
  std::lock_guard<std::mutex> g(t.mu);
  fmm::Launcher L;
  L.timer = &t;
  return fmm::launch_forward(a, L) == hipSuccess ? FMM_OK : FMM_ERR_HIP;
}

// ------------------------------------------------------------------ one-launch path
// Mode: 0 never, 1 wherever it applies (default), 2 wherever it applies but
// with every workgroup forming its slice's state itself (no exchange).
std::atomic<int>& one_launch_mode() {
  static std::atomic<int> m{1};
  return m;
}

// Epochs of the one-launch path's stamps (56 bits, formed on the device): this
// call's number in bits 32-55, from a random start, and in bits 0-31 a random
// per-process offset to which each launch adds its dispatch id.  Eager calls
// differ in the call number, replays of a captured graph (frozen arguments)
// in the dispatch id; the random parts make a match with stale stamps left in
// memory by another process unlikely.
unsigned long long next_epoch() {
  static const unsigned long long offset = [] {
    std::random_device rd;
    return (unsigned long long)rd();
  }();
  static std::atomic<unsigned long long> n{[] {
    std::random_device rd;
    return (unsigned long long)rd();
  }()};
  const unsigned long long c = n.fetch_add(1, std::memory_order_relaxed) & 0xffffffull;
  return (c << 32) | (offset & 0xffffffffull);
}

// Workgroups of k_band_fused that fit on the current device at once (two per CU).
int resident_fused_workgroups() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  if (dev >= 0 && dev < 64) {
    const int c = cache[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  if (dev >= 0 && dev < 64) cache[dev].store(2 * cus, std::memory_order_relaxed);
  return 2 * cus;
}

fmm::LaunchArgs make_args(const void* q, const void* k, const void* v, void* out, int B, int H,
                          int N, int d, int band_k, int rank, int causal, const float* w_near,
                          const float* w_far, int dtype, int far_norm, void* ws, const Plan& p,
                          void* stream) {
  fmm::LaunchArgs a;
  a.far_norm = far_norm;
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.w_near = w_near;
  a.w_far = w_far;
  a.B = B;
  a.H = H;
  a.N = N;
  a.d = d;
  // a half-width of N already covers every key; clamping keeps row +/- k in int range
  a.band_k = band_k < N ? band_k : N;
  a.rank = rank;
  a.causal = causal;
  a.dtype = dtype;
  a.stream = stream;
  a.ws = (float*)ws;
  a.nseg = p.nseg;
  a.L = p.L;
  a.nseg_apply = p.nseg_apply;
  a.L_apply = p.L_apply;
  const int mode = one_launch_mode().load(std::memory_order_relaxed);
  if (p.fused_g > 0 && mode != 0 && far_norm == FMM_FAR_NORM_PER_MAP &&
      (long long)B * H * p.fused_g <= resident_fused_workgroups()) {
    a.fused_g = p.fused_g;
    a.exchange = mode == 2 ? 0 : 1;
    a.epoch = next_epoch();
  }
  return a;
}

// Adds the one-launch path's workspace to a plan (the larger of the two).
void add_fused(Plan& p, long long bh, int G, int d, int rank) {
  p.fused_g = G;
  if (G <= 0 || p.ws_bytes == 0) return;
  const size_t f = fmm::fused_layout(bh, G, (long long)rank * d * (d + 1)).total;
  if (f > p.ws_bytes) p.ws_bytes = f;
}

Plan plan_for(int B, int H, int N, int d, int band_k, int rank, int causal, int dtype) {
  const int kc = band_k < N ? band_k : N;
  const int apply_tm = fmm::band_pair_applies(dtype, d, kc, causal, N) ? fmm::pair_tile_rows()
                                                                    : fmm::tile_rows();
  Plan p = make_plan(B, H, N, d, rank, dtype == FMM_DTYPE_BF16 ? 2 : 4, apply_tm);
  const long long bh = (long long)B * H;
  add_fused(p, bh, fmm::fused_groups(dtype, d, kc, rank, causal, bh, N, kFusedPlanWorkgroups), d,
            rank);
  return p;
}


int run(const void* q, const void* k, const void* v, void* out, int B, int H, int N, int d,
        int band_k, int rank, int causal, const float* w_near, const float* w_far, int dtype,
        int far_norm, void* ws, size_t ws_bytes, bool own_ws, void* stream) {
  int st = validate(q, k, v, out, B, H, N, d, band_k, rank, causal, w_near, w_far, dtype,
                    far_norm);
  if (st != FMM_OK) return st;
  const Plan p = plan_for(B, H, N, d, band_k, rank, causal, dtype);
  if (p.ws_bytes == 0) return FMM_ERR_UNSUPPORTED;
  fmm::LaunchArgs a = make_args(q, k, v, out, B, H, N, d, band_k, rank, causal, w_near, w_far,
                                dtype, far_norm, nullptr, p, stream);
  st = check_launch(a);
  if (st != FMM_OK) return st;
  std::unique_lock<std::mutex> ws_lock(ws_mutex(), std::defer_lock);
  if (own_ws) {
    ws_lock.lock();
    st = acquire_ws_locked(stream, p.ws_bytes, &ws);
    if (st != FMM_OK) return st;
  } else {
    if (!ws || (uintptr_t)ws % 256) return FMM_ERR_INVALID_ARG;
    if (ws_bytes < p.ws_bytes) return FMM_ERR_OOM;
  }
  a.ws = (float*)ws;
  return launch_now(a);
}

// ------------------------------------------------------------------ backward
struct BwdPlan {
  Plan p;
  size_t off_dpart, off_rowstat, off_rowfar, off_dwpart, total;
};

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Workspace of the backward pass: the forward state records (as the forward
// plan), the dS records of the same shape, per-row softmax statistics and far
// quotients, and per-segment blend sums.  0 when it cannot exist.
BwdPlan bwd_plan(int B, int H, int N, int d, int rank, int dtype) {
  BwdPlan b;
  b.p = make_plan(B, H, N, d, rank, dtype == FMM_DTYPE_BF16 ? 2 : 4, fmm::tile_rows());
  b.total = 0;
  if (b.p.ws_bytes == 0) return b;
  typedef unsigned __int128 u128;
  const u128 bhn = (u128)B * H * N;
  const u128 rowstat = (u128)align256((size_t)std::min<u128>(bhn * 12, SIZE_MAX / 8));
  const u128 rowfar = (u128)align256((size_t)std::min<u128>(bhn * rank * 8, SIZE_MAX / 8));
  const u128 dwp = align256((size_t)B * H * b.p.nseg * 8);
  const u128 tot = 2 * (u128)b.p.ws_bytes + rowstat + rowfar + dwp;
  if (tot > (u128)(SIZE_MAX / 4)) return b;
  b.off_dpart = b.p.ws_bytes;
  b.off_rowstat = 2 * b.p.ws_bytes;
  b.off_rowfar = b.off_rowstat + (size_t)rowstat;
  b.off_dwpart = b.off_rowfar + (size_t)rowfar;
  b.total = (size_t)tot;
  return b;
}

void fill_bwd_args(fmm::BwdArgs& a, const BwdPlan& bp, void* ws, int B, int H) {
  const uintptr_t w = reinterpret_cast<uintptr_t>(ws);
  const size_t rec = (size_t)a.rank * a.d * (a.d + 1);
  const size_t fin_off = (size_t)B * H * bp.p.nseg * rec * sizeof(float);
  a.part = reinterpret_cast<float*>(w);
  a.fin = reinterpret_cast<float*>(w + fin_off);
  a.dpart = reinterpret_cast<float*>(w + bp.off_dpart);
  a.dfin = reinterpret_cast<float*>(w + bp.off_dpart + fin_off);
  a.rowstat = reinterpret_cast<float*>(w + bp.off_rowstat);
  a.rowfar = reinterpret_cast<float*>(w + bp.off_rowfar);
  a.dwpart = reinterpret_cast<float*>(w + bp.off_dwpart);
}

int run_backward(const void* q, const void* k, const void* v, const void* dout, void* dq,
                 void* dk, void* dv, float* dw_near, float* dw_far, int B, int H, int N, int d,
                 int band_k, int rank, int causal, const float* w_near, const float* w_far,
                 int dtype, int far_norm, void* stream) {
  // the inputs as in the forward (dout takes the place of out for the checks)
  int st = validate(q, k, v, dq, B, H, N, d, band_k, rank, causal, w_near, w_far, dtype,
                    far_norm);
  if (st != FMM_OK) return st;
  if (!dout || !dk || !dv || !dw_near || !dw_far) return FMM_ERR_INVALID_ARG;
  const size_t es = dtype == FMM_DTYPE_BF16 ? 2 : 4;
  const size_t bytes = (size_t)B * H * N * d * es;  // fits: validate checked it
  for (const void* p : {dout, (const void*)dk, (const void*)dv})
    if ((uintptr_t)p % 16) return FMM_ERR_INVALID_ARG;
  if ((uintptr_t)dw_near % 4 || (uintptr_t)dw_far % 4) return FMM_ERR_INVALID_ARG;
  // gradients overlap neither the inputs nor one another
  const void* ins[4] = {q, k, v, dout};
  void* outs[3] = {dq, dk, dv};
  for (void* o : outs)
    for (const void* i : ins)
      if (overlaps(o, i, bytes)) return FMM_ERR_INVALID_ARG;
  if (overlaps(dq, dk, bytes) || overlaps(dq, dv, bytes) || overlaps(dk, dv, bytes))
    return FMM_ERR_INVALID_ARG;
  if (overlaps(dw_near, dw_far, (size_t)H * 4)) return FMM_ERR_INVALID_ARG;
  const BwdPlan bp = bwd_plan(B, H, N, d, rank, dtype);
  if (bp.total == 0) return FMM_ERR_UNSUPPORTED;
  fmm::LaunchArgs fa = make_args(q, k, v, dq, B, H, N, d, band_k, rank, causal, w_near, w_far,
                                 dtype, FMM_FAR_NORM_PER_MAP, nullptr, bp.p, stream);
  fmm::BwdArgs ba;
  ba.q = q;
  ba.k = k;
  ba.v = v;
  ba.dout = dout;
  ba.dq = dq;
  ba.dk = dk;
  ba.dv = dv;
  ba.dw_near = dw_near;
  ba.dw_far = dw_far;
  ba.w_near = w_near;
  ba.w_far = w_far;
  ba.B = B;
  ba.H = H;
  ba.N = N;
  ba.d = d;
  ba.band_k = fa.band_k;
  ba.rank = rank;
  ba.causal = causal;
  ba.dtype = dtype;
  ba.far_norm = far_norm;
  ba.stream = stream;
  ba.nseg = bp.p.nseg;
  ba.L = bp.p.L;
  fill_bwd_args(ba, bp, nullptr, B, H);
  EventTimer& t = timer();
  {
    std::lock_guard<std::mutex> g(t.mu);
    fmm::Launcher dry;
    dry.timer = &t;
    dry.dry = true;
    if (fmm::launch_state_only(fa, dry) != hipSuccess ||
        fmm::launch_backward_tail(ba, dry) != hipSuccess)
      return dry.err == hipErrorInvalidConfiguration ? FMM_ERR_UNSUPPORTED : FMM_ERR_HIP;
  }
  std::lock_guard<std::mutex> wl(ws_mutex());
  void* ws = nullptr;
  st = acquire_ws_locked(stream, bp.total, &ws);
  if (st != FMM_OK) return st;
  fa.ws = (float*)ws;
  fill_bwd_args(ba, bp, ws, B, H);
  std::lock_guard<std::mutex> g(t.mu);
  fmm::Launcher L;
  L.timer = &t;
  if (fmm::launch_state_only(fa, L) != hipSuccess) return FMM_ERR_HIP;
  return fmm::launch_backward_tail(ba, L) == hipSuccess ? FMM_OK : FMM_ERR_HIP;
}

// ------------------------------------------------------------------ layer
std::mutex& blas_mutex() {
  static std::mutex* m = new std::mutex();
  return *m;
}

// rocBLAS handle of the current device (created once per device).
void* blas_handle() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  static std::map<int, void*>* handles = new std::map<int, void*>();
  void*& h = (*handles)[dev];
  if (!h) h = fmm::layer_blas_handle_create();
  return h;
}

int run_layer(const void* x, const void* w_qkv, const void* w_out, void* y, int B, int N, int E,
              int H, int band_k, int rank, int causal, const float* w_near, const float* w_far,
              int dtype, void* stream) {
  if (!x || !w_qkv || !w_out || !y || !w_near || !w_far) return FMM_ERR_INVALID_ARG;
  if (B < 1 || N < 1 || E < 1 || H < 1 || band_k < 0 || E % H) return FMM_ERR_INVALID_ARG;
  if (causal != 0 && causal != 1) return FMM_ERR_INVALID_ARG;
  if (dtype != FMM_DTYPE_F32 && dtype != FMM_DTYPE_BF16) return FMM_ERR_UNSUPPORTED;
  const int d = E / H;
  if (!supported(d, rank)) return FMM_ERR_UNSUPPORTED;
  const size_t es = dtype == FMM_DTYPE_BF16 ? 2 : 4;
  typedef unsigned __int128 u128;
  const u128 tokens = (u128)B * N;
  if (tokens > (u128)INT32_MAX || (u128)3 * E > (u128)INT32_MAX) return FMM_ERR_UNSUPPORTED;
  const u128 xbytes = tokens * E * es;
  if (xbytes * 8 > (u128)INT64_MAX) return FMM_ERR_INVALID_ARG;
  for (const void* p : {x, w_qkv, w_out, (const void*)y})
    if ((uintptr_t)p % 16) return FMM_ERR_INVALID_ARG;
  if ((uintptr_t)w_near % 4 || (uintptr_t)w_far % 4) return FMM_ERR_INVALID_ARG;
  const size_t xb = (size_t)xbytes, wq = (size_t)E * 3 * E * es, wo = (size_t)E * E * es;
  if (overlaps2(y, xb, x, xb) || overlaps2(y, xb, w_qkv, wq) || overlaps2(y, xb, w_out, wo))
    return FMM_ERR_INVALID_ARG;
  // workspace: qkv, q, k, v, o, merged heads, then the operator's records
  // (with the library's own projection kernels only q, k, v and o are used)
  const Plan p = plan_for(B, H, N, d, band_k, rank, causal, dtype);
  if (p.ws_bytes == 0) return FMM_ERR_UNSUPPORTED;
  const bool own_proj = fmm::layer_proj_applies(dtype, E);
  const size_t seg = align256(xb);
  const size_t off_qkv = 0, off_q = 3 * seg, off_k = 4 * seg, off_v = 5 * seg, off_o = 6 * seg,
               off_m = 7 * seg, off_ws = 8 * seg;
  const size_t total = off_ws + p.ws_bytes;
  auto at = [](void* base, size_t off) {
    return reinterpret_cast<void*>(reinterpret_cast<uintptr_t>(base) + off);
  };
  fmm::LaunchArgs a = make_args(at(nullptr, off_q), at(nullptr, off_k), at(nullptr, off_v),
                                at(nullptr, off_o), B, H, N, d, band_k, rank, causal, w_near,
                                w_far, dtype, FMM_FAR_NORM_PER_MAP, nullptr, p, stream);
  int st = check_launch(a);
  if (st != FMM_OK) return st;
  {
    EventTimer& t = timer();
    std::lock_guard<std::mutex> g(t.mu);
    fmm::Launcher dry;
    dry.timer = &t;
    dry.dry = true;
    // (the dry passes record their result in dry.err)
    if (own_proj) {
      (void)fmm::launch_layer_proj(dry, true, nullptr, nullptr, nullptr, nullptr, nullptr, B, N,
                                   H, d, (hipStream_t)stream);
      (void)fmm::launch_layer_proj(dry, false, nullptr, nullptr, nullptr, nullptr, nullptr, B, N,
                                   H, d, (hipStream_t)stream);
    } else {
      (void)fmm::launch_layer_copy(dry, true, dtype, nullptr, nullptr, nullptr, nullptr, B, N, H,
                                   d, (hipStream_t)stream);
      (void)fmm::launch_layer_copy(dry, false, dtype, nullptr, nullptr, nullptr, nullptr, B, N,
                                   H, d, (hipStream_t)stream);
    }
    if (dry.err != hipSuccess)
      return dry.err == hipErrorInvalidConfiguration ? FMM_ERR_UNSUPPORTED : FMM_ERR_HIP;
  }
  std::lock_guard<std::mutex> bl(blas_mutex());
  void* hdl = blas_handle();
  if (!hdl) return FMM_ERR_HIP;
  std::lock_guard<std::mutex> wl(ws_mutex());
  void* ws = nullptr;
  st = acquire_ws_locked(stream, total, &ws);
  if (st != FMM_OK) return st;
  a.q = at(ws, off_q);
  a.k = at(ws, off_k);
  a.v = at(ws, off_v);
  a.out = at(ws, off_o);
  a.ws = (float*)at(ws, off_ws);
  const int M = B * N;
  if (own_proj) {
    EventTimer& t = timer();
    std::lock_guard<std::mutex> g(t.mu);
    fmm::Launcher L;
    L.timer = &t;
    if (fmm::launch_layer_proj(L, true, x, w_qkv, at(ws, off_q), at(ws, off_k), at(ws, off_v), B,
                               N, H, d, (hipStream_t)stream) != hipSuccess ||
        fmm::launch_forward(a, L) != hipSuccess ||
        fmm::launch_layer_proj(L, false, at(ws, off_o), w_out, y, nullptr, nullptr, B, N, H, d,
                               (hipStream_t)stream) != hipSuccess)
      return FMM_ERR_HIP;
    return FMM_OK;
  }
  if (fmm::layer_gemm(hdl, stream, dtype, x, w_qkv, at(ws, off_qkv), M, E, 3 * E) != hipSuccess)
    return FMM_ERR_HIP;
  EventTimer& t = timer();
  std::lock_guard<std::mutex> g(t.mu);
  fmm::Launcher L;
  L.timer = &t;
  if (fmm::launch_layer_copy(L, true, dtype, at(ws, off_qkv), at(ws, off_q), at(ws, off_k),
                             at(ws, off_v), B, N, H, d, (hipStream_t)stream) != hipSuccess ||
      fmm::launch_forward(a, L) != hipSuccess ||
      fmm::launch_layer_copy(L, false, dtype, at(ws, off_o), at(ws, off_m), nullptr, nullptr, B,
                             N, H, d, (hipStream_t)stream) != hipSuccess)
    return FMM_ERR_HIP;
  if (fmm::layer_gemm(hdl, stream, dtype, at(ws, off_m), w_out, y, M, E, E) != hipSuccess)
    return FMM_ERR_HIP;
  return FMM_OK;
}

// Backward of the layer: the forward recomputed through rocBLAS and the
// operator (qkv, the heads q, k, v, their outputs o and the merged rows m),
// then dm = dy W_out^T, dW_out = m^T dy, the operator's backward for the
// heads' share of dm, dqkv = [dq | dk | dv] per token, dx = dqkv W_qkv^T and
// dW_qkv = x^T dqkv.
int run_layer_backward(const void* x, const void* w_qkv, const void* w_out, const void* dy,
                       void* dx, void* dw_qkv, void* dw_out, float* dw_near, float* dw_far,
                       int B, int N, int E, int H, int band_k, int rank, int causal,
                       const float* w_near, const float* w_far, int dtype, void* stream) {
  if (!x || !w_qkv || !w_out || !dy || !dx || !dw_qkv || !dw_out || !dw_near || !dw_far ||
      !w_near || !w_far)
    return FMM_ERR_INVALID_ARG;
  if (B < 1 || N < 1 || E < 1 || H < 1 || band_k < 0 || E % H) return FMM_ERR_INVALID_ARG;
  if (causal != 0 && causal != 1) return FMM_ERR_INVALID_ARG;
  if (dtype != FMM_DTYPE_F32 && dtype != FMM_DTYPE_BF16) return FMM_ERR_UNSUPPORTED;
  const int d = E / H;
  if (!supported(d, rank)) return FMM_ERR_UNSUPPORTED;
  const size_t es = dtype == FMM_DTYPE_BF16 ? 2 : 4;
  typedef unsigned __int128 u128;
  const u128 tokens = (u128)B * N;
  if (tokens > (u128)INT32_MAX || (u128)3 * E > (u128)INT32_MAX) return FMM_ERR_UNSUPPORTED;
  const u128 xbytes = tokens * E * es;
  if (xbytes * 16 > (u128)INT64_MAX) return FMM_ERR_INVALID_ARG;
  for (const void* p : {x, w_qkv, w_out, dy, (const void*)dx, (const void*)dw_qkv,
                        (const void*)dw_out})
    if ((uintptr_t)p % 16) return FMM_ERR_INVALID_ARG;
  if ((uintptr_t)w_near % 4 || (uintptr_t)w_far % 4 || (uintptr_t)dw_near % 4 ||
      (uintptr_t)dw_far % 4)
    return FMM_ERR_INVALID_ARG;
  const size_t xb = (size_t)xbytes, wq = (size_t)E * 3 * E * es, wo = (size_t)E * E * es;
  // outputs overlap neither the inputs nor one another
  const void* ins[4] = {x, w_qkv, w_out, dy};
  const size_t in_b[4] = {xb, wq, wo, xb};
  void* outs[3] = {dx, dw_qkv, dw_out};
  const size_t out_b[3] = {xb, wq, wo};
  for (int o = 0; o < 3; ++o) {
    for (int i = 0; i < 4; ++i)
      if (overlaps2(outs[o], out_b[o], ins[i], in_b[i])) return FMM_ERR_INVALID_ARG;
    for (int o2 = o + 1; o2 < 3; ++o2)
      if (overlaps2(outs[o], out_b[o], outs[o2], out_b[o2])) return FMM_ERR_INVALID_ARG;
  }
  if (overlaps(dw_near, dw_far, (size_t)H * 4)) return FMM_ERR_INVALID_ARG;
  // workspace: qkv (later dqkv), q, k, v, o, m, dm, do, dq, dk, dv, then the
  // forward operator's and the backward's records
  const Plan p = plan_for(B, H, N, d, band_k, rank, causal, dtype);
  const BwdPlan bp = bwd_plan(B, H, N, d, rank, dtype);
  if (p.ws_bytes == 0 || bp.total == 0) return FMM_ERR_UNSUPPORTED;
  const size_t seg = align256(xb);
  const size_t off_qkv = 0, off_q = 3 * seg, off_k = 4 * seg, off_v = 5 * seg, off_o = 6 * seg,
               off_m = 7 * seg, off_dm = 8 * seg, off_do = 9 * seg, off_dq = 10 * seg,
               off_dk = 11 * seg, off_dv = 12 * seg, off_fws = 13 * seg,
               off_bws = off_fws + align256(p.ws_bytes),
               off_wg = off_bws + align256(bp.total);
  const int Mtok = B * N;  // fits: checked above
  const size_t total = off_wg + align256(fmm::layer_wgrad_scratch_bytes(Mtok, E, 3 * E));
  auto at = [](void* base, size_t off) {
    return reinterpret_cast<void*>(reinterpret_cast<uintptr_t>(base) + off);
  };
  fmm::LaunchArgs a = make_args(at(nullptr, off_q), at(nullptr, off_k), at(nullptr, off_v),
                                at(nullptr, off_o), B, H, N, d, band_k, rank, causal, w_near,
                                w_far, dtype, FMM_FAR_NORM_PER_MAP, nullptr, p, stream);
  int st = check_launch(a);
  if (st != FMM_OK) return st;
  fmm::LaunchArgs fa = make_args(at(nullptr, off_q), at(nullptr, off_k), at(nullptr, off_v),
                                 at(nullptr, off_dq), B, H, N, d, band_k, rank, causal, w_near,
                                 w_far, dtype, FMM_FAR_NORM_PER_MAP, nullptr, bp.p, stream);
  fmm::BwdArgs ba;
  ba.q = at(nullptr, off_q);
  ba.k = at(nullptr, off_k);
  ba.v = at(nullptr, off_v);
  ba.dout = at(nullptr, off_do);
  ba.dq = at(nullptr, off_dq);
  ba.dk = at(nullptr, off_dk);
  ba.dv = at(nullptr, off_dv);
  ba.dw_near = dw_near;
  ba.dw_far = dw_far;
  ba.w_near = w_near;
  ba.w_far = w_far;
  ba.B = B;
  ba.H = H;
  ba.N = N;
  ba.d = d;
  ba.band_k = fa.band_k;
  ba.rank = rank;
  ba.causal = causal;
  ba.dtype = dtype;
  ba.stream = stream;
  ba.nseg = bp.p.nseg;
  ba.L = bp.p.L;
  fill_bwd_args(ba, bp, nullptr, B, H);
  hipStream_t s = (hipStream_t)stream;
  {
    EventTimer& t = timer();
    std::lock_guard<std::mutex> g(t.mu);
    fmm::Launcher dry;
    dry.timer = &t;
    dry.dry = true;
    (void)fmm::launch_layer_copy(dry, true, dtype, nullptr, nullptr, nullptr, nullptr, B, N, H, d,
                                 s);
    (void)fmm::launch_layer_copy(dry, false, dtype, nullptr, nullptr, nullptr, nullptr, B, N, H,
                                 d, s);
    (void)fmm::launch_layer_split1(dry, dtype, nullptr, nullptr, B, N, H, d, s);
    (void)fmm::launch_layer_merge_part(dry, dtype, nullptr, nullptr, 0, B, N, H, d, s);
    if (dry.err == hipSuccess) (void)fmm::launch_state_only(fa, dry);
    if (dry.err == hipSuccess) (void)fmm::launch_backward_tail(ba, dry);
    if (dry.err == hipSuccess)
      (void)fmm::layer_wgrad(nullptr, dry, stream, dtype, nullptr, nullptr, nullptr, Mtok, E,
                             3 * E, nullptr);
    if (dry.err != hipSuccess)
      return dry.err == hipErrorInvalidConfiguration ? FMM_ERR_UNSUPPORTED : FMM_ERR_HIP;
  }
  std::lock_guard<std::mutex> bl(blas_mutex());
  void* hdl = blas_handle();
  if (!hdl) return FMM_ERR_HIP;
  std::lock_guard<std::mutex> wl(ws_mutex());
  void* ws = nullptr;
  st = acquire_ws_locked(stream, total, &ws);
  if (st != FMM_OK) return st;
  a.q = ba.q = at(ws, off_q);
  a.k = ba.k = at(ws, off_k);
  a.v = ba.v = at(ws, off_v);
  a.out = at(ws, off_o);
  a.ws = (float*)at(ws, off_fws);
  fa.q = a.q;
  fa.k = a.k;
  fa.v = a.v;
  fa.ws = (float*)at(ws, off_bws);
  ba.dout = at(ws, off_do);
  ba.dq = at(ws, off_dq);
  ba.dk = at(ws, off_dk);
  ba.dv = at(ws, off_dv);
  fill_bwd_args(ba, bp, at(ws, off_bws), B, H);
  const int M = B * N;
  EventTimer& t = timer();
  // the forward: qkv, the heads, the operator, the merged rows
  if (fmm::layer_gemm(hdl, stream, dtype, x, w_qkv, at(ws, off_qkv), M, E, 3 * E) != hipSuccess)
    return FMM_ERR_HIP;
  {
    std::lock_guard<std::mutex> g(t.mu);
    fmm::Launcher L;
    L.timer = &t;
    if (fmm::launch_layer_copy(L, true, dtype, at(ws, off_qkv), at(ws, off_q), at(ws, off_k),
                               at(ws, off_v), B, N, H, d, s) !=
            hipSuccess ||
        fmm::launch_forward(a, L) != hipSuccess ||
        fmm::launch_layer_copy(L, false, dtype, a.out, at(ws, off_m), nullptr, nullptr, B, N, H,
                               d, s) != hipSuccess)
      return FMM_ERR_HIP;
  }
  // dm = dy W_out^T, dW_out = m^T dy
  float* wg = reinterpret_cast<float*>(at(ws, off_wg));
  if (fmm::layer_gemm(hdl, stream, dtype, dy, w_out, at(ws, off_dm), M, E, E, false, true) !=
      hipSuccess)
    return FMM_ERR_HIP;
  {
    std::lock_guard<std::mutex> g(t.mu);
    fmm::Launcher L;
    L.timer = &t;
    if (fmm::layer_wgrad(hdl, L, stream, dtype, at(ws, off_m), dy, dw_out, M, E, E, wg) !=
        hipSuccess)
      return FMM_ERR_HIP;
  }
  // the operator's backward on the heads' share of dm, then dqkv per token
  {
    std::lock_guard<std::mutex> g(t.mu);
    fmm::Launcher L;
    L.timer = &t;
    if (fmm::launch_layer_split1(L, dtype, at(ws, off_dm), at(ws, off_do), B, N, H, d, s) !=
            hipSuccess ||
        fmm::launch_state_only(fa, L) != hipSuccess ||
        fmm::launch_backward_tail(ba, L) != hipSuccess ||
        fmm::launch_layer_merge_part(L, dtype, ba.dq, at(ws, off_qkv), 0, B, N, H, d, s) !=
            hipSuccess ||
        fmm::launch_layer_merge_part(L, dtype, ba.dk, at(ws, off_qkv), 1, B, N, H, d, s) !=
            hipSuccess ||
        fmm::launch_layer_merge_part(L, dtype, ba.dv, at(ws, off_qkv), 2, B, N, H, d, s) !=
            hipSuccess)
      return FMM_ERR_HIP;
  }
  // dx = dqkv W_qkv^T, dW_qkv = x^T dqkv
  if (fmm::layer_gemm(hdl, stream, dtype, at(ws, off_qkv), w_qkv, dx, M, 3 * E, E, false,
                      true) != hipSuccess)
    return FMM_ERR_HIP;
  std::lock_guard<std::mutex> g(t.mu);
  fmm::Launcher L;
  L.timer = &t;
  return fmm::layer_wgrad(hdl, L, stream, dtype, x, at(ws, off_qkv), dw_qkv, M, E, 3 * E, wg) ==
                 hipSuccess
             ? FMM_OK
             : FMM_ERR_HIP;
}

// ------------------------------------------------------------------ fast weight
int run_fastweight(const void* q, const void* k, const void* v, const float* beta, void* out,
                   int B, int H, int N, int d, int band_k, int n_linear, const float* w_near,
                   const float* w_far, int dtype, void* stream) {
  int st = validate(q, k, v, out, B, H, N, d, band_k, 1, 1, w_near, w_far, dtype,
                    FMM_FAR_NORM_PER_MAP);
  if (st != FMM_OK) return st;
  if (!beta || (uintptr_t)beta % 4 || (n_linear != 0 && n_linear != 1))
    return FMM_ERR_INVALID_ARG;
  const Plan p = plan_for(B, H, N, d, band_k, 1, 1, dtype);
  if (p.ws_bytes == 0) return FMM_ERR_UNSUPPORTED;
  // the operator's records, then H floats of -inf that remove its linear
  // far part when n_linear = 0, then p(k) and p(q) of every position for the
  // narrow scan
  const size_t pre_bytes = fmm::fast_weight_pre_bytes(B, H, N, d);
  if (pre_bytes > SIZE_MAX / 4) return FMM_ERR_UNSUPPORTED;
  const size_t total = p.ws_bytes + align256((size_t)H * 4) + align256(pre_bytes);
  fmm::LaunchArgs a = make_args(q, k, v, out, B, H, N, d, band_k, 1, 1, w_near, w_far, dtype,
                                FMM_FAR_NORM_PER_MAP, nullptr, p, stream);
  fmm::FwArgs f;
  f.q = q;
  f.k = k;
  f.v = v;
  f.beta = beta;
  f.out = out;
  f.w_far = w_far;
  f.B = B;
  f.H = H;
  f.N = N;
  f.d = d;
  f.dtype = dtype;
  f.stream = stream;
  EventTimer& t = timer();
  {
    std::lock_guard<std::mutex> g(t.mu);
    fmm::Launcher dry;
    dry.timer = &t;
    dry.dry = true;
    // (the dry pass only checks grids: the scratch pointer just selects the
    // kernels)
    static float dry_placeholder;
    if (fmm::launch_forward(a, dry) != hipSuccess ||
        fmm::launch_fast_weight_pre(dry, f, pre_bytes ? &dry_placeholder : nullptr) !=
            hipSuccess)
      return dry.err == hipErrorInvalidConfiguration ? FMM_ERR_UNSUPPORTED : FMM_ERR_HIP;
  }
  std::lock_guard<std::mutex> wl(ws_mutex());
  void* ws = nullptr;
  st = acquire_ws_locked(stream, total, &ws);
  if (st != FMM_OK) return st;
  a.ws = (float*)ws;
  float* minus_inf =
      reinterpret_cast<float*>(reinterpret_cast<uintptr_t>(ws) + p.ws_bytes);
  float* pre = pre_bytes ? reinterpret_cast<float*>(reinterpret_cast<uintptr_t>(ws) + p.ws_bytes +
                                                    align256((size_t)H * 4))
                         : nullptr;
  std::lock_guard<std::mutex> g(t.mu);
  fmm::Launcher L;
  L.timer = &t;
  if (!n_linear) {
    if (fmm::launch_fill(L, minus_inf, H, -INFINITY, stream) != hipSuccess) return FMM_ERR_HIP;
    a.w_far = minus_inf;
  }
  if (fmm::launch_forward(a, L) != hipSuccess) return FMM_ERR_HIP;
  return fmm::launch_fast_weight_pre(L, f, pre) == hipSuccess ? FMM_OK : FMM_ERR_HIP;
}

// Backward of the fast-weight operator: the operator's backward at rank 1,
// causal (the near field, and the linear far part when n_linear = 1; with
// n_linear = 0 its far part is removed by -inf logits), then the fast-weight
// kernel, which adds its gradients to dq, dk, dv, writes dbeta and adds its
// share to dw_far.
int run_backward_fastweight(const void* q, const void* k, const void* v, const float* beta,
                            const void* dout, void* dq, void* dk, void* dv, float* dbeta,
                            float* dw_near, float* dw_far, int B, int H, int N, int d,
                            int band_k, int n_linear, const float* w_near, const float* w_far,
                            int dtype, void* stream) {
  int st = validate(q, k, v, dq, B, H, N, d, band_k, 1, 1, w_near, w_far, dtype,
                    FMM_FAR_NORM_PER_MAP);
  if (st != FMM_OK) return st;
  if (!dout || !dk || !dv || !dw_near || !dw_far || !beta || !dbeta) return FMM_ERR_INVALID_ARG;
  if (n_linear != 0 && n_linear != 1) return FMM_ERR_INVALID_ARG;
  const size_t es = dtype == FMM_DTYPE_BF16 ? 2 : 4;
  const size_t bytes = (size_t)B * H * N * d * es;  // fits: validate checked it
  for (const void* p : {dout, (const void*)dk, (const void*)dv})
    if ((uintptr_t)p % 16) return FMM_ERR_INVALID_ARG;
  if ((uintptr_t)dw_near % 4 || (uintptr_t)dw_far % 4 || (uintptr_t)beta % 4 ||
      (uintptr_t)dbeta % 4)
    return FMM_ERR_INVALID_ARG;
  const void* ins[4] = {q, k, v, dout};
  void* outs[3] = {dq, dk, dv};
  for (void* o : outs)
    for (const void* i : ins)
      if (overlaps(o, i, bytes)) return FMM_ERR_INVALID_ARG;
  if (overlaps(dq, dk, bytes) || overlaps(dq, dv, bytes) || overlaps(dk, dv, bytes))
    return FMM_ERR_INVALID_ARG;
  const size_t nb = (size_t)B * H * N * 4;
  for (const void* o : {(const void*)dq, (const void*)dk, (const void*)dv})
    if (overlaps2(dbeta, nb, o, bytes)) return FMM_ERR_INVALID_ARG;
  if (overlaps2(dbeta, nb, beta, nb) || overlaps(dw_near, dw_far, (size_t)H * 4))
    return FMM_ERR_INVALID_ARG;
  const BwdPlan bp = bwd_plan(B, H, N, d, 1, dtype);
  if (bp.total == 0) return FMM_ERR_UNSUPPORTED;
  // after the backward's workspace: W_i and z_i of every step, the per-slice
  // sums, H floats of -inf
  typedef unsigned __int128 u128;
  const u128 wst = (u128)B * H * N * d * d * 4, zst = (u128)B * H * N * d * 4;
  // then, for d = 16 and 32, p(k), p(q) and their inverse sums of every
  // position for the narrow sweeps
  const size_t pre_bytes = fmm::fast_weight_backward_pre_bytes(B, H, N, d);
  const u128 tot = (u128)bp.total + align256((size_t)std::min<u128>(wst, SIZE_MAX / 8)) +
                   align256((size_t)std::min<u128>(zst, SIZE_MAX / 8)) +
                   align256((size_t)B * H * 4) + align256((size_t)H * 4) +
                   align256(std::min<size_t>(pre_bytes, SIZE_MAX / 8));
  if (tot > (u128)(SIZE_MAX / 4)) return FMM_ERR_UNSUPPORTED;
  const size_t off_w = bp.total, off_z = off_w + align256((size_t)wst);
  const size_t off_g = off_z + align256((size_t)zst), off_m = off_g + align256((size_t)B * H * 4);
  const size_t off_p = off_m + align256((size_t)H * 4);
  fmm::LaunchArgs fa = make_args(q, k, v, dq, B, H, N, d, band_k, 1, 1, w_near, w_far, dtype,
                                 FMM_FAR_NORM_PER_MAP, nullptr, bp.p, stream);
  fmm::BwdArgs ba;
  ba.q = q;
  ba.k = k;
  ba.v = v;
  ba.dout = dout;
  ba.dq = dq;
  ba.dk = dk;
  ba.dv = dv;
  ba.dw_near = dw_near;
  ba.dw_far = dw_far;
  ba.w_near = w_near;
  ba.w_far = w_far;
  ba.B = B;
  ba.H = H;
  ba.N = N;
  ba.d = d;
  ba.band_k = fa.band_k;
  ba.rank = 1;
  ba.causal = 1;
  ba.dtype = dtype;
  ba.stream = stream;
  ba.nseg = bp.p.nseg;
  ba.L = bp.p.L;
  fill_bwd_args(ba, bp, nullptr, B, H);
  fmm::FwBwdArgs fb;
  fb.q = q;
  fb.k = k;
  fb.v = v;
  fb.beta = beta;
  fb.dout = dout;
  fb.dq = dq;
  fb.dk = dk;
  fb.dv = dv;
  fb.dbeta = dbeta;
  fb.dw_far = dw_far;
  fb.w_far = w_far;
  fb.wst = fb.zst = fb.gfw = nullptr;
  fb.B = B;
  fb.H = H;
  fb.N = N;
  fb.d = d;
  fb.dtype = dtype;
  fb.stream = stream;
  EventTimer& t = timer();
  {
    std::lock_guard<std::mutex> g(t.mu);
    fmm::Launcher dry;
    dry.timer = &t;
    dry.dry = true;
    static float dry_placeholder;  // (selects the kernels; the dry pass reads nothing)
    if (fmm::launch_state_only(fa, dry) != hipSuccess ||
        fmm::launch_backward_tail(ba, dry) != hipSuccess ||
        fmm::launch_fast_weight_backward_pre(dry, fb, pre_bytes ? &dry_placeholder : nullptr) !=
            hipSuccess)
      return dry.err == hipErrorInvalidConfiguration ? FMM_ERR_UNSUPPORTED : FMM_ERR_HIP;
  }
  std::lock_guard<std::mutex> wl(ws_mutex());
  void* ws = nullptr;
  st = acquire_ws_locked(stream, (size_t)tot, &ws);
  if (st != FMM_OK) return st;
  const uintptr_t w = reinterpret_cast<uintptr_t>(ws);
  fa.ws = (float*)ws;
  fill_bwd_args(ba, bp, ws, B, H);
  fb.wst = reinterpret_cast<float*>(w + off_w);
  fb.zst = reinterpret_cast<float*>(w + off_z);
  fb.gfw = reinterpret_cast<float*>(w + off_g);
  float* minus_inf = reinterpret_cast<float*>(w + off_m);
  float* pre = pre_bytes ? reinterpret_cast<float*>(w + off_p) : nullptr;
  std::lock_guard<std::mutex> g(t.mu);
  fmm::Launcher L;
  L.timer = &t;
  if (!n_linear) {
    if (fmm::launch_fill(L, minus_inf, H, -INFINITY, stream) != hipSuccess) return FMM_ERR_HIP;
    fa.w_far = minus_inf;
    ba.w_far = minus_inf;
  }
  if (fmm::launch_state_only(fa, L) != hipSuccess) return FMM_ERR_HIP;
  if (fmm::launch_backward_tail(ba, L) != hipSuccess) return FMM_ERR_HIP;
  return fmm::launch_fast_weight_backward_pre(L, fb, pre) == hipSuccess ? FMM_OK : FMM_ERR_HIP;
}

}  // namespace

namespace fmm {

int validate_forward(const void* q, const void* k, const void* v, void* out, int B, int H,
                     int N, int d, int band_k, int rank, int causal, const float* w_near,
                     const float* w_far, int dtype) {
  return validate(q, k, v, out, B, H, N, d, band_k, rank, causal, w_near, w_far, dtype,
                  FMM_FAR_NORM_PER_MAP);
}

size_t forward_workspace_bytes(int B, int H, int N, int d, int band_k, int rank, int causal,
                               int dtype) {
  return plan_for(B, H, N, d, band_k, rank, causal, dtype).ws_bytes;
}

int forward_with_workspace(const void* q, const void* k, const void* v, void* out, int B, int H,
                           int N, int d, int band_k, int rank, int causal, const float* w_near,
                           const float* w_far, int dtype, void* ws, size_t ws_bytes,
                           void* stream) {
  return run(q, k, v, out, B, H, N, d, band_k, rank, causal, w_near, w_far, dtype,
             FMM_FAR_NORM_PER_MAP, ws, ws_bytes, false, stream);
}

}  // namespace fmm

extern "C" {

int fmm_attn_forward(const void* q, const void* k, const void* v, void* out, int B, int H,
                     int N, int d, int band_k, int rank, int causal, const float* w_near,
                     const float* w_far, void* stream) {
  return run(q, k, v, out, B, H, N, d, band_k, rank, causal, w_near, w_far, FMM_DTYPE_F32,
             FMM_FAR_NORM_PER_MAP, nullptr, 0, true, stream);
}

int fmm_attn_forward_bf16(const void* q, const void* k, const void* v, void* out, int B, int H,
                          int N, int d, int band_k, int rank, int causal, const float* w_near,
                          const float* w_far, void* stream) {
  return run(q, k, v, out, B, H, N, d, band_k, rank, causal, w_near, w_far, FMM_DTYPE_BF16,
             FMM_FAR_NORM_PER_MAP, nullptr, 0, true, stream);
}

int fmm_attn_forward_ex(const void* q, const void* k, const void* v, void* out, int B, int H,
                        int N, int d, int band_k, int rank, int causal, const float* w_near,
                        const float* w_far, int dtype, int far_norm, void* stream) {
  return run(q, k, v, out, B, H, N, d, band_k, rank, causal, w_near, w_far, dtype, far_norm,
             nullptr, 0, true, stream);
}

int fmm_attn_backward(const void* q, const void* k, const void* v, const void* dout, void* dq,
                      void* dk, void* dv, float* dw_near, float* dw_far, int B, int H, int N,
                      int d, int band_k, int rank, int causal, const float* w_near,
                      const float* w_far, int dtype, void* stream) {
  return run_backward(q, k, v, dout, dq, dk, dv, dw_near, dw_far, B, H, N, d, band_k, rank,
                      causal, w_near, w_far, dtype, FMM_FAR_NORM_PER_MAP, stream);
}

int fmm_attn_backward_ex(const void* q, const void* k, const void* v, const void* dout,
                         void* dq, void* dk, void* dv, float* dw_near, float* dw_far, int B,
                         int H, int N, int d, int band_k, int rank, int causal,
                         const float* w_near, const float* w_far, int dtype, int far_norm,
                         void* stream) {
  return run_backward(q, k, v, dout, dq, dk, dv, dw_near, dw_far, B, H, N, d, band_k, rank,
                      causal, w_near, w_far, dtype, far_norm, stream);
}

int fmm_attn_layer_backward(const void* x, const void* w_qkv, const void* w_out, const void* dy,
                            void* dx, void* dw_qkv, void* dw_out, float* dw_near, float* dw_far,
                            int B, int N, int E, int H, int band_k, int rank, int causal,
                            const float* w_near, const float* w_far, int dtype, void* stream) {
  return run_layer_backward(x, w_qkv, w_out, dy, dx, dw_qkv, dw_out, dw_near, dw_far, B, N, E, H,
                            band_k, rank, causal, w_near, w_far, dtype, stream);
}

int fmm_attn_backward_fastweight(const void* q, const void* k, const void* v, const float* beta,
                                 const void* dout, void* dq, void* dk, void* dv, float* dbeta,
                                 float* dw_near, float* dw_far, int B, int H, int N, int d,
                                 int band_k, int n_linear, const float* w_near,
                                 const float* w_far, int dtype, void* stream) {
  return run_backward_fastweight(q, k, v, beta, dout, dq, dk, dv, dbeta, dw_near, dw_far, B, H,
                                 N, d, band_k, n_linear, w_near, w_far, dtype, stream);
}

int fmm_attn_layer_forward(const void* x, const void* w_qkv, const void* w_out, void* y, int B,
                           int N, int E, int H, int band_k, int rank, int causal,
                           const float* w_near, const float* w_far, int dtype, void* stream) {
  return run_layer(x, w_qkv, w_out, y, B, N, E, H, band_k, rank, causal, w_near, w_far, dtype,
                   stream);
}

int fmm_attn_forward_fastweight(const void* q, const void* k, const void* v, const float* beta,
                                void* out, int B, int H, int N, int d, int band_k, int n_linear,
                                const float* w_near, const float* w_far, int dtype,
                                void* stream) {
  return run_fastweight(q, k, v, beta, out, B, H, N, d, band_k, n_linear, w_near, w_far, dtype,
                        stream);
}

size_t fmm_attn_workspace_bytes(int B, int H, int N, int d, int rank, int causal) {
  if (B < 1 || H < 1 || N < 1 || (causal != 0 && causal != 1) || !supported(d, rank)) return 0;
  // the plan depends on the element size only through the segment length
  // floor; report the larger of the two dtypes' needs
  const int tm = fmm::tile_rows();
  Plan a = make_plan(B, H, N, d, rank, 2, tm), b = make_plan(B, H, N, d, rank, 4, tm);
  // the one-launch path (bf16, any band it takes)
  const long long bh = (long long)B * H;
  add_fused(a, bh,
            fmm::fused_groups(FMM_DTYPE_BF16, d, 0, rank, causal, bh, N, kFusedPlanWorkgroups),
            d, rank);
  return a.ws_bytes > b.ws_bytes ? a.ws_bytes : b.ws_bytes;
}

int fmm_attn_set_one_launch(int mode) {
  if (mode < 0 || mode > 2) return -1;
  return one_launch_mode().exchange(mode);
}

int fmm_attn_forward_ws(const void* q, const void* k, const void* v, void* out, int B, int H,
                        int N, int d, int band_k, int rank, int causal, const float* w_near,
                        const float* w_far, int dtype, void* workspace, size_t ws_bytes,
                        void* stream) {
  return run(q, k, v, out, B, H, N, d, band_k, rank, causal, w_near, w_far, dtype,
             FMM_FAR_NORM_PER_MAP, workspace, ws_bytes, false, stream);
}

const char* fmm_attn_status_string(int status) {
  switch (status) {
    case FMM_OK: return "FMM_OK: success";
    case FMM_ERR_INVALID_ARG:
      return "FMM_ERR_INVALID_ARG: null, negative, misaligned or overlapping argument";
    case FMM_ERR_UNSUPPORTED:
      return "FMM_ERR_UNSUPPORTED: d must be 16, 32, 64 or 128 and rank 1, 2 or 3, within the "
             "dispatch limits";
    case FMM_ERR_HIP: return "FMM_ERR_HIP: a HIP runtime call or kernel launch failed";
    case FMM_ERR_OOM: return "FMM_ERR_OOM: workspace allocation failed or workspace too small";
    case FMM_ERR_SCRATCH:
      return "FMM_ERR_SCRATCH: the shape needs more scratch than the fixed no-allocation array";
    default: return "unknown fmm_attn status";
  }
}

void fmm_attn_release_workspace(void) {
  std::lock_guard<std::mutex> g(ws_mutex());
  int cur = 0;
  const bool have_cur = hipGetDevice(&cur) == hipSuccess;
  for (auto& kv : ws_map()) {
    if (!kv.second.ptr) continue;
    (void)hipSetDevice(kv.first.first);
    (void)hipDeviceSynchronize();
    (void)hipFree(kv.second.ptr);
  }
  ws_map().clear();
  if (have_cur) (void)hipSetDevice(cur);
}

int fmm_attn_version(void) { return kVersion; }

int fmm_attn_kernel_timing(int enable) {
  EventTimer& t = timer();
  std::lock_guard<std::mutex> g(t.mu);
  t.enabled = enable != 0;
  return FMM_OK;
}

int fmm_attn_kernel_timing_read(int kernel, double* total_ms, long long* launches) {
  if (kernel < 0 || kernel >= FMM_KERNEL_COUNT || !total_ms || !launches)
    return FMM_ERR_INVALID_ARG;
  EventTimer& t = timer();
  std::lock_guard<std::mutex> g(t.mu);
  double sum = 0.0;
  long long n = 0;
  int st = FMM_OK;
  for (auto& pr : t.pending[kernel]) {
    float ms = 0.f;
    if (hipEventSynchronize(pr.second) != hipSuccess ||
        hipEventElapsedTime(&ms, pr.first, pr.second) != hipSuccess)
      st = FMM_ERR_HIP;
    sum += ms;
    ++n;
    t.pool.push_back(pr.first);
    t.pool.push_back(pr.second);
  }
  t.pending[kernel].clear();
  *total_ms = sum;
  *launches = n;
  return st;
}

}  // extern "C"
