// C ABI of libcats: argument validation (all on the host, before any HIP
// call), workspace carving, kernel dispatch and the optional kernel timer.
#include <hip/hip_runtime.h>

#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <random>
#include <string>
#include <vector>

#include "cats.h"
#include "internal.hpp"

namespace {

thread_local std::string g_last_error;

cats_status fail(cats_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

cats_status hip_fail(hipError_t e, const char* what) {
  return fail(CATS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Debug mode: with CATS_SYNC_CHECK set to anything but "" or "0" in the
// environment, every enqueue-only call synchronises its stream after its
// launches and reports an asynchronous failure (a kernel fault, a launch
// error) as CATS_ERR_HIP from the call that launched it.  A stream under
// graph capture cannot be synchronised; such calls are left as they are.
bool sync_check_on() {
  const char* e = std::getenv("CATS_SYNC_CHECK");
  return e && e[0] && !(e[0] == '0' && e[1] == 0);
}

cats_status sync_check(void* stream, const char* what) {
  if (!sync_check_on()) return CATS_OK;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cs) == hipSuccess && cs != hipStreamCaptureStatusNone) return CATS_OK;
  hipError_t e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, what);
  e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, what);
  return CATS_OK;
}

cats_status checked(cats_status st, void* stream, const char* what) {
  return st != CATS_OK ? st : sync_check(stream, what);
}

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

constexpr size_t kAlign = 256;
constexpr size_t kRadixWords = 260;
constexpr int kMaxBatchTile = 8;

// Workspace regions.  The radix-select scratch always sits at offset 0;
// the MLP region and the calibration activations share the space after it
// (no call uses both).
struct FwdLayout {
  size_t partial, seg_j, seg_mask, seg_v, seg_h, seg_cnt, end;
};

size_t radix_bytes() { return round_up(kRadixWords * sizeof(uint32_t), kAlign); }

// Neuron groups and column tiles of the batched down-projection.
int down_ct(int d) { return (d + cats::kDownCols - 1) / cats::kDownCols; }
int down_ng(int d, int m) {
  const int G = cats::fused_grid(m);
  const int ng = cats::kFusedBlocks / down_ct(d);
  return ng < 1 ? 1 : (ng > G ? G : ng);
}

// Layout for calls of up to B rows: the partial sums of either path (the
// fused kernel's per-block partials of one pass of up to kMaxBatchTile rows,
// or the batched path's per-group partials of all B rows) and the segment
// lists for B rows.
FwdLayout fwd_layout(int d, int m, int B) {
  const int G = cats::fused_grid(m);
  const int bp = B < kMaxBatchTile ? B : kMaxBatchTile;
  size_t parts = (size_t)G * bp;
  const size_t parts_b = (size_t)down_ng(d, m) * B;
  if (parts_b > parts) parts = parts_b;
  FwdLayout L;
  size_t o = radix_bytes();
  L.partial = o;
  o = round_up(o + parts * d * sizeof(float), kAlign);
  L.seg_j = o;
  o = round_up(o + (size_t)m * sizeof(int32_t), kAlign);
  L.seg_mask = o;
  o = round_up(o + (size_t)m * sizeof(uint32_t), kAlign);
  L.seg_v = o;
  o = round_up(o + (size_t)B * m * sizeof(float), kAlign);
  L.seg_h = o;
  o = round_up(o + (size_t)B * m * sizeof(float), kAlign);
  L.seg_cnt = o;
  o = round_up(o + (size_t)cats::kFusedBlocks * sizeof(int32_t), kAlign);
  L.end = o;
  return L;
}

// Two [B x d] fp32 buffers a stack ping-pongs its residual stream through
// (placed after the forward region of the largest layer).
size_t stack_rows_bytes(int d, int B) { return 2 * round_up((size_t)B * d * sizeof(float), kAlign); }

size_t calib_bytes(int64_t nvalues) {
  return radix_bytes() + round_up((size_t)nvalues * sizeof(float), kAlign);
}

bool d_ok(int32_t d, int32_t wdtype) {
  if (d <= 0 || d % 8 != 0) return false;
  return d <= (wdtype == CATS_BF16 ? CATS_MAX_D_BF16 : CATS_MAX_D_F32);
}

cats_status check_layer(const cats_layer* L) {
  if (!L) return fail(CATS_ERR_NULL, "layer is NULL");
  if (L->wdtype != CATS_F32 && L->wdtype != CATS_BF16)
    return fail(CATS_ERR_DTYPE, "unknown weight dtype %d", (int)L->wdtype);
  if (!d_ok(L->d, L->wdtype))
    return fail(CATS_ERR_SHAPE, "d=%d must be a positive multiple of 8 and at most %d", (int)L->d,
                L->wdtype == CATS_BF16 ? CATS_MAX_D_BF16 : CATS_MAX_D_F32);
  if (L->m <= 0 || L->m > CATS_MAX_M)
    return fail(CATS_ERR_SHAPE, "m=%d must be in [1, %d]", (int)L->m, CATS_MAX_M);
  if (!L->w_gate_t || !L->w_up_t || !L->w_down) return fail(CATS_ERR_NULL, "a weight pointer is NULL");
  if (!aligned(L->w_gate_t, 16) || !aligned(L->w_up_t, 16) || !aligned(L->w_down, 16))
    return fail(CATS_ERR_ALIGN, "weight pointers must be 16-byte aligned");
  const uint64_t mat = (uint64_t)L->m * L->d * (L->wdtype == CATS_BF16 ? 2 : 4);
  if (mat > CATS_MAX_MATRIX_BYTES)
    return fail(CATS_ERR_SHAPE, "each weight matrix must be at most %llu bytes (m*d*%d = %llu)",
                (unsigned long long)CATS_MAX_MATRIX_BYTES, L->wdtype == CATS_BF16 ? 2 : 4,
                (unsigned long long)mat);
  return CATS_OK;
}

cats_status check_ws(const void* ws, size_t ws_bytes, size_t need) {
  if (!ws) return fail(CATS_ERR_WORKSPACE, "workspace is NULL");
  if (!aligned(ws, kAlign)) return fail(CATS_ERR_ALIGN, "workspace must be 256-byte aligned");
  if (ws_bytes < need)
    return fail(CATS_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  return CATS_OK;
}

int batch_tile(int rows) {
  int bt = 1;
  while (bt < rows) bt *= 2;
  return bt;
}

// Shared body of forward and dense.
// norm: x is RMSNorm'ed (unit gain, eps) inside the fused kernel first.
cats_status run_mlp(const cats_layer* L, const float* x, int32_t B, float t, bool dense,
                    const float* residual, float* y, const cats_forward_aux* aux, void* ws,
                    size_t ws_bytes, void* stream, bool norm = false, float eps = 0.f,
                    const float* vin = nullptr, const float* vin_t = nullptr) {
  cats_status st = check_layer(L);
  if (st != CATS_OK) return st;
  if (!x || !y) return fail(CATS_ERR_NULL, "x or y is NULL");
  if (B < 1 || B > CATS_MAX_BATCH) return fail(CATS_ERR_SHAPE, "B=%d outside [1, %d]", (int)B, CATS_MAX_BATCH);
  if (!aligned(x, 16) || !aligned(y, 16) || (residual && !aligned(residual, 16)))
    return fail(CATS_ERR_ALIGN, "x, y and residual must be 16-byte aligned");
  if (std::isnan(t) || t < 0.f) return fail(CATS_ERR_RANGE, "t must be >= 0 (got %g)", (double)t);
  const bool want_aux = aux && (aux->active_idx || aux->active_cnt || aux->active_v || aux->active_h);
  if (want_aux && ((aux->active_idx && !aligned(aux->active_idx, 4)) ||
                   (aux->active_cnt && !aligned(aux->active_cnt, 4)) ||
                   (aux->active_v && !aligned(aux->active_v, 4)) ||
                   (aux->active_h && !aligned(aux->active_h, 4))))
    return fail(CATS_ERR_ALIGN, "aux outputs must be 4-byte aligned");
  const int bf16 = L->wdtype == CATS_BF16;
  const int d = L->d, m = L->m;
  const int nch = cats::fused_nch(bf16, d);
  const int bt_max = cats::fused_bt_max(bf16, nch);
  const int rows_per_pass = B < bt_max ? B : bt_max;
  const FwdLayout lay = fwd_layout(d, m, B);
  // the full cats_workspace_bytes(d, m, B, 0), stack rows included, so one
  // size rule holds for every call
  st = check_ws(ws, ws_bytes, lay.end + stack_rows_bytes(d, B));
  if (st != CATS_OK) return st;

  char* w = static_cast<char*>(ws);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int G = cats::fused_grid(m);
  if (!vin && bf16 && B >= cats::kBatchedMinRows && cats::batched_ks(d) > 0) {
    // all rows in one pass: gate/up on the matrix cores, down by column tiles
    cats::BatchedArgs ba;
    ba.wg = L->w_gate_t;
    ba.wu = L->w_up_t;
    ba.x = x;
    ba.B = B;
    ba.d = d;
    ba.m = m;
    ba.t = dense ? 0.f : t;
    ba.norm = norm ? 1 : 0;
    ba.eps = eps;
    ba.seg_j = reinterpret_cast<int*>(w + lay.seg_j);
    ba.seg_mask = reinterpret_cast<uint32_t*>(w + lay.seg_mask);
    ba.seg_v = reinterpret_cast<float*>(w + lay.seg_v);
    ba.seg_h = reinterpret_cast<float*>(w + lay.seg_h);
    ba.seg_cnt = reinterpret_cast<int*>(w + lay.seg_cnt);
    hipError_t e = cats::launch_gateup(dense, want_aux, ba, G, s);
    if (e != hipSuccess) return hip_fail(e, "gate/up launch");
    cats::DownArgs da;
    da.wd = L->w_down;
    da.partial = reinterpret_cast<float*>(w + lay.partial);
    da.seg_j = ba.seg_j;
    da.seg_h = ba.seg_h;
    da.seg_cnt = ba.seg_cnt;
    da.B = B;
    da.d = d;
    da.m = m;
    da.G = G;
    da.NG = down_ng(d, m);
    da.CT = down_ct(d);
    e = cats::launch_down_mfma(da, s);
    if (e != hipSuccess) return hip_fail(e, "down-projection launch");
    cats::ReduceArgs ra;
    ra.partial = da.partial;
    ra.G = da.NG;
    ra.Gseg = G;
    ra.sum_y = 1;
    ra.B = B;
    ra.d = d;
    ra.m = m;
    ra.residual = residual;
    ra.y = y;
    ra.aux = want_aux ? 1 : 0;
    ra.seg_j = ba.seg_j;
    ra.seg_mask = ba.seg_mask;
    ra.seg_v = ba.seg_v;
    ra.seg_h = ba.seg_h;
    ra.seg_cnt = ba.seg_cnt;
    ra.active_idx = want_aux ? aux->active_idx : nullptr;
    ra.active_cnt = want_aux ? aux->active_cnt : nullptr;
    ra.active_v = want_aux ? aux->active_v : nullptr;
    ra.active_h = want_aux ? aux->active_h : nullptr;
    e = cats::launch_reduce(ra, s);
    if (e != hipSuccess) return hip_fail(e, "reduce launch");
    return CATS_OK;
  }
  for (int b0 = 0; b0 < B; b0 += rows_per_pass) {
    const int bp = (B - b0) < rows_per_pass ? (B - b0) : rows_per_pass;
    cats::FusedArgs fa;
    fa.wg = L->w_gate_t;
    fa.wu = L->w_up_t;
    fa.wd = L->w_down;
    fa.x = x + (size_t)b0 * d;
    fa.B = bp;
    fa.d = d;
    fa.m = m;
    fa.t = dense ? 0.f : t;
    fa.norm = norm ? 1 : 0;
    fa.eps = eps;
    fa.vin = vin ? vin + (size_t)b0 * m : nullptr;
    fa.vin_t = vin_t ? vin_t + b0 : nullptr;
    fa.partial = reinterpret_cast<float*>(w + lay.partial);
    fa.aux = want_aux ? 1 : 0;
    fa.seg_j = reinterpret_cast<int*>(w + lay.seg_j);
    fa.seg_mask = reinterpret_cast<uint32_t*>(w + lay.seg_mask);
    fa.seg_v = reinterpret_cast<float*>(w + lay.seg_v);
    fa.seg_h = reinterpret_cast<float*>(w + lay.seg_h);
    fa.seg_cnt = reinterpret_cast<int*>(w + lay.seg_cnt);
    const int bt = batch_tile(bp);
    hipError_t e;
    if (vin)
      e = bf16 ? cats::launch_fused_bf16_topk(nch, bt, fa.aux != 0, fa, G, s)
               : cats::launch_fused_f32_topk(nch, bt, fa.aux != 0, fa, G, s);
    else if (bf16)
      e = dense ? cats::launch_fused_bf16_dense(nch, bt, fa, G, s)
          : fa.aux ? cats::launch_fused_bf16_cats_aux(nch, bt, fa, G, s)
                   : cats::launch_fused_bf16_cats(nch, bt, fa, G, s);
    else
      e = dense ? cats::launch_fused_f32_dense(nch, bt, fa, G, s)
          : fa.aux ? cats::launch_fused_f32_cats_aux(nch, bt, fa, G, s)
                   : cats::launch_fused_f32_cats(nch, bt, fa, G, s);
    if (e != hipSuccess) return hip_fail(e, "fused MLP launch");

    cats::ReduceArgs ra;
    ra.partial = fa.partial;
    ra.G = G;
    ra.Gseg = G;
    ra.sum_y = 1;
    ra.B = bp;
    ra.d = d;
    ra.m = m;
    ra.residual = residual ? residual + (size_t)b0 * d : nullptr;
    ra.y = y + (size_t)b0 * d;
    ra.aux = fa.aux;
    ra.seg_j = fa.seg_j;
    ra.seg_mask = fa.seg_mask;
    ra.seg_v = fa.seg_v;
    ra.seg_h = fa.seg_h;
    ra.seg_cnt = fa.seg_cnt;
    ra.active_idx = (want_aux && aux->active_idx) ? aux->active_idx + (size_t)b0 * m : nullptr;
    ra.active_cnt = (want_aux && aux->active_cnt) ? aux->active_cnt + b0 : nullptr;
    ra.active_v = (want_aux && aux->active_v) ? aux->active_v + (size_t)b0 * m : nullptr;
    ra.active_h = (want_aux && aux->active_h) ? aux->active_h + (size_t)b0 * m : nullptr;
    e = cats::launch_reduce(ra, s);
    if (e != hipSuccess) return hip_fail(e, "reduce launch");
  }
  return CATS_OK;
}

int64_t cutoff_rank(int64_t n, double k) {
  if (k == 0.0) return 0;
  double r = std::ceil(k * (double)n - 1e-6);
  if (r < 1) r = 1;
  if (r > (double)n) r = (double)n;
  return (int64_t)r;
}

cats_status select_threshold(const float* acts, int64_t n, double k, void* ws, hipStream_t s,
                             float* t_out) {
  const int64_t r = cutoff_rank(n, k);
  if (r == 0) {
    *t_out = 0.f;
    return CATS_OK;
  }
  uint32_t* sc = static_cast<uint32_t*>(ws);
  hipError_t e = cats::launch_radix_select(acts, n, r, sc, s);
  if (e != hipSuccess) return hip_fail(e, "radix select launch");
  uint32_t bits = 0;
  e = hipMemcpyAsync(&bits, sc + 256, sizeof(bits), hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return hip_fail(e, "threshold copy");
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "stream synchronize");
  float t;
  memcpy(&t, &bits, sizeof(t));
  *t_out = t;
  return CATS_OK;
}

// ---- kernel timer ---------------------------------------------------------
struct TimerState {
  std::mutex mu;
  bool on = false;
  std::vector<std::string> names;
  std::vector<int64_t> launches;
  std::vector<double> total_ms;
  struct Pending {
    int name;
    hipEvent_t a, b;
  };
  std::vector<Pending> pending;
  std::vector<hipEvent_t> pool;
};

TimerState& timer_state() {
  static TimerState* st = new TimerState();  // lives until process exit
  return *st;
}

int timer_name_index(TimerState& T, const char* name) {
  for (size_t i = 0; i < T.names.size(); ++i)
    if (T.names[i] == name) return (int)i;
  T.names.emplace_back(name);
  T.launches.push_back(0);
  T.total_ms.push_back(0.0);
  return (int)T.names.size() - 1;
}

hipError_t timer_flush_locked(TimerState& T) {
  hipError_t first = hipSuccess;
  for (auto& p : T.pending) {
    hipError_t e = hipEventSynchronize(p.b);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.a, p.b);
    if (e == hipSuccess) {
      T.launches[p.name] += 1;
      T.total_ms[p.name] += ms;
    } else if (first == hipSuccess) {
      first = e;
    }
    T.pool.push_back(p.a);
    T.pool.push_back(p.b);
  }
  T.pending.clear();
  return first;
}

hipEvent_t timer_event_locked(TimerState& T) {
  if (!T.pool.empty()) {
    hipEvent_t e = T.pool.back();
    T.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

}  // namespace

namespace cats {
cats_status report_error(cats_status st, const char* msg) { return fail(st, "%s", msg); }
}  // namespace cats

static_assert(CATS_MAX_M == cats::kMaxNeurons, "CATS_MAX_M must match the kernel's neuron capacity");

namespace cats {

int fused_nch(int wdtype_bf16, int d) {
  const int need = (d + chunk_elems(wdtype_bf16) - 1) / chunk_elems(wdtype_bf16);
  static const int inst[] = {1, 2, 4, 8, 10, 16};
  for (int n : inst)
    if (n >= need) return n;
  return 16;
}

int fused_bt_max(int wdtype_bf16, int nch) {
  const int row_bytes = nch * chunk_elems(wdtype_bf16) * (int)sizeof(float);
  int bt = kMaxBatchTile;
  while (bt > 1 && bt * row_bytes > kXLdsBytes) bt /= 2;
  return bt;
}

int fused_grid(int m) { return m < kFusedBlocks ? m : kFusedBlocks; }

KernelTimer::KernelTimer(const char* name, hipStream_t) {
  TimerState& T = timer_state();
  std::lock_guard<std::mutex> lk(T.mu);
  if (!T.on) return;
  if (T.pending.size() >= 4096) timer_flush_locked(T);
  TimerState::Pending p;
  p.name = timer_name_index(T, name);
  p.a = timer_event_locked(T);
  p.b = timer_event_locked(T);
  if (!p.a || !p.b) return;
  T.pending.push_back(p);
  a_ = p.a;
  b_ = p.b;
}

}  // namespace cats

extern "C" {

int32_t cats_version(void) { return CATS_VERSION; }

const char* cats_status_string(cats_status s) {
  switch (s) {
    case CATS_OK: return "ok";
    case CATS_ERR_NULL: return "null pointer";
    case CATS_ERR_SHAPE: return "unsupported shape";
    case CATS_ERR_RANGE: return "argument out of range";
    case CATS_ERR_DTYPE: return "unknown dtype";
    case CATS_ERR_ALIGN: return "misaligned pointer";
    case CATS_ERR_WORKSPACE: return "workspace missing or too small";
    case CATS_ERR_HIP: return "HIP runtime error";
    case CATS_ERR_UNIMPLEMENTED: return "not implemented";
  }
  return "unknown status";
}

const char* cats_last_error(void) { return g_last_error.c_str(); }

size_t cats_workspace_bytes(int32_t d, int32_t m, int32_t max_batch, int64_t max_calib_values) {
  if (d <= 0 || d % 8 != 0 || d > CATS_MAX_D_BF16 || m <= 0 || m > CATS_MAX_M || max_batch < 1 ||
      max_batch > CATS_MAX_BATCH || max_calib_values < 0)
    return 0;
  const size_t fwd = fwd_layout(d, m, max_batch).end + stack_rows_bytes(d, max_batch);
  const size_t cal = calib_bytes(max_calib_values);
  return fwd > cal ? fwd : cal;
}

cats_status cats_pack_weights(const void* w, void* w_t, int32_t rows, int32_t cols, int32_t dtype,
                              void* stream) {
  if (!w || !w_t) return fail(CATS_ERR_NULL, "w or w_t is NULL");
  if (dtype != CATS_F32 && dtype != CATS_BF16) return fail(CATS_ERR_DTYPE, "unknown dtype %d", (int)dtype);
  if (rows <= 0 || cols <= 0 || rows > (65535 * 32)) return fail(CATS_ERR_SHAPE, "bad shape %d x %d", (int)rows, (int)cols);
  const int eb = dtype == CATS_BF16 ? 2 : 4;
  if (!aligned(w, eb) || !aligned(w_t, eb)) return fail(CATS_ERR_ALIGN, "w and w_t must be element-aligned");
  const size_t bytes = (size_t)rows * cols * eb;
  const char* a = static_cast<const char*>(w);
  const char* b = static_cast<const char*>(w_t);
  if (a < b + bytes && b < a + bytes) return fail(CATS_ERR_RANGE, "w and w_t overlap");
  hipError_t e = cats::launch_transpose(w, w_t, rows, cols, eb, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "transpose launch");
  return sync_check(stream, "cats_pack_weights");
}

cats_status cats_calib_activations(const cats_layer* layer, const float* x, int32_t N, float* acts,
                                   void* stream) {
  cats_status st = check_layer(layer);
  if (st != CATS_OK) return st;
  if (!x || !acts) return fail(CATS_ERR_NULL, "x or acts is NULL");
  if (N <= 0 || N > 4 * 1024 * 1024) return fail(CATS_ERR_SHAPE, "N=%d out of range", (int)N);
  if (!aligned(x, 16) || !aligned(acts, 4)) return fail(CATS_ERR_ALIGN, "x must be 16-byte and acts 4-byte aligned");
  hipError_t e = cats::launch_calib_acts(layer->wdtype == CATS_BF16, x, layer->w_gate_t, N, layer->d,
                                         layer->m, acts, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "calibration activations launch");
  return sync_check(stream, "cats_calib_activations");
}

cats_status cats_threshold_from_acts(const float* acts, int64_t n, double sparsity, void* ws,
                                     size_t ws_bytes, void* stream, float* t_out) {
  if (!acts || !t_out) return fail(CATS_ERR_NULL, "acts or t_out is NULL");
  if (n <= 0 || n > (int64_t)0xffffffffll) return fail(CATS_ERR_SHAPE, "n=%lld out of range", (long long)n);
  if (!std::isfinite(sparsity) || sparsity < 0.0 || sparsity > 1.0)
    return fail(CATS_ERR_RANGE, "sparsity must be in [0, 1]");
  if (!aligned(acts, 4)) return fail(CATS_ERR_ALIGN, "acts must be 4-byte aligned");
  if (sparsity == 0.0) {
    *t_out = 0.f;
    return CATS_OK;
  }
  cats_status st = check_ws(ws, ws_bytes, radix_bytes());
  if (st != CATS_OK) return st;
  return select_threshold(acts, n, sparsity, ws, static_cast<hipStream_t>(stream), t_out);
}

cats_status cats_calibrate_threshold(const cats_layer* layer, const float* calib_x, int32_t N,
                                     double sparsity, void* ws, size_t ws_bytes, void* stream,
                                     float* t_out) {
  cats_status st = check_layer(layer);
  if (st != CATS_OK) return st;
  if (!calib_x || !t_out) return fail(CATS_ERR_NULL, "calib_x or t_out is NULL");
  if (N <= 0 || N > 4 * 1024 * 1024) return fail(CATS_ERR_SHAPE, "N=%d out of range", (int)N);
  if (!aligned(calib_x, 16)) return fail(CATS_ERR_ALIGN, "calib_x must be 16-byte aligned");
  if (!std::isfinite(sparsity) || sparsity < 0.0 || sparsity > 1.0)
    return fail(CATS_ERR_RANGE, "sparsity must be in [0, 1]");
  const int64_t n = (int64_t)N * layer->m;
  if (n > (int64_t)0xffffffffll) return fail(CATS_ERR_SHAPE, "N*m=%lld too large", (long long)n);
  if (sparsity == 0.0) {
    *t_out = 0.f;
    return CATS_OK;
  }
  st = check_ws(ws, ws_bytes, calib_bytes(n));
  if (st != CATS_OK) return st;
  float* acts = reinterpret_cast<float*>(static_cast<char*>(ws) + radix_bytes());
  const hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = cats::launch_calib_acts(layer->wdtype == CATS_BF16, calib_x, layer->w_gate_t, N,
                                         layer->d, layer->m, acts, s);
  if (e != hipSuccess) return hip_fail(e, "calibration activations launch");
  return select_threshold(acts, n, sparsity, ws, s, t_out);
}

cats_status cats_mlp_forward(const cats_layer* layer, const float* x, int32_t B, float t,
                             const float* residual, float* y, const cats_forward_aux* aux, void* ws,
                             size_t ws_bytes, void* stream) {
  return checked(run_mlp(layer, x, B, t, false, residual, y, aux, ws, ws_bytes, stream), stream, "cats_mlp_forward");
}

cats_status cats_mlp_dense(const cats_layer* layer, const float* x, int32_t B, const float* residual,
                           float* y, void* ws, size_t ws_bytes, void* stream) {
  return checked(run_mlp(layer, x, B, 0.f, true, residual, y, nullptr, ws, ws_bytes, stream), stream,
                 "cats_mlp_dense");
}

cats_status cats_stack_forward(const cats_layer* layers, int32_t L, const float* t, const float* x0,
                               int32_t B, float eps, float* x_out, float* x_all,
                               const cats_forward_aux* aux, void* ws, size_t ws_bytes,
                               void* stream) {
  if (!layers) return fail(CATS_ERR_NULL, "layers is NULL");
  if (!x0 || !x_out) return fail(CATS_ERR_NULL, "x0 or x_out is NULL");
  if (L < 1 || L > CATS_MAX_LAYERS) return fail(CATS_ERR_SHAPE, "L=%d outside [1, %d]", (int)L, CATS_MAX_LAYERS);
  if (B < 1 || B > CATS_MAX_BATCH) return fail(CATS_ERR_SHAPE, "B=%d outside [1, %d]", (int)B, CATS_MAX_BATCH);
  if (!std::isfinite(eps) || eps < 0.f) return fail(CATS_ERR_RANGE, "eps must be finite and >= 0");
  if (!t && aux) return fail(CATS_ERR_RANGE, "aux outputs need thresholds (t is NULL: dense stack)");
  if (!aligned(x0, 16) || !aligned(x_out, 16) || (x_all && !aligned(x_all, 16)))
    return fail(CATS_ERR_ALIGN, "x0, x_out and x_all must be 16-byte aligned");
  const int d = layers[0].d;
  size_t fwd_end = 0;
  for (int l = 0; l < L; ++l) {
    cats_status st = check_layer(&layers[l]);
    if (st != CATS_OK) return fail(st, "layer %d: %s", l, g_last_error.c_str());
    if (layers[l].d != d) return fail(CATS_ERR_SHAPE, "layer %d has d=%d, layer 0 has d=%d", l, (int)layers[l].d, d);
    if (t && (std::isnan(t[l]) || t[l] < 0.f)) return fail(CATS_ERR_RANGE, "t[%d] must be >= 0 (got %g)", l, (double)t[l]);
    const size_t e = fwd_layout(d, layers[l].m, B).end;
    if (e > fwd_end) fwd_end = e;
  }
  const size_t rows = (size_t)B * d;
  const char* xo = reinterpret_cast<const char*>(x_out);
  const char* xi = reinterpret_cast<const char*>(x0);
  if (xo < xi + rows * 4 && xi < xo + rows * 4) return fail(CATS_ERR_RANGE, "x_out overlaps x0");
  cats_status st = check_ws(ws, ws_bytes, fwd_end + stack_rows_bytes(d, B));
  if (st != CATS_OK) return st;

  const hipStream_t s = static_cast<hipStream_t>(stream);
  float* pp[2] = {reinterpret_cast<float*>(static_cast<char*>(ws) + fwd_end),
                  reinterpret_cast<float*>(static_cast<char*>(ws) + fwd_end +
                                           round_up(rows * sizeof(float), kAlign))};
  if (x_all) {
    hipError_t e = hipMemcpyAsync(x_all, x0, rows * sizeof(float), hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "x_all[0] copy");
  }
  const float* cur = x0;
  for (int l = 0; l < L; ++l) {
    // the layer's output: x_all[l+1] when kept, the caller's x_out for the
    // last layer, otherwise the ping-pong buffer cur does not occupy
    float* dst = x_all ? x_all + (size_t)(l + 1) * rows : (l == L - 1 ? x_out : pp[l & 1]);
    st = run_mlp(&layers[l], cur, B, t ? t[l] : 0.f, t == nullptr, cur, dst, aux ? &aux[l] : nullptr,
                 ws, ws_bytes, stream, true, eps);
    if (st != CATS_OK) return fail(st, "layer %d: %s", l, g_last_error.c_str());
    cur = dst;
  }
  if (x_all) {
    hipError_t e = hipMemcpyAsync(x_out, cur, rows * sizeof(float), hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "x_out copy");
  }
  return sync_check(stream, "cats_stack_forward");
}

namespace {
// Workspace of cats_sparse_input_gemv: the groups' partial sums, the
// column tiles' tickets and the segment lists over the d input channels.
struct GemvLayout {
  size_t partial, tickets, seg_j, seg_mask, seg_v, seg_h, seg_cnt, end;
  int NG, CT;
};

GemvLayout gemv_layout(int d, int n, int B) {
  GemvLayout L;
  L.CT = (n + cats::kSparseCols - 1) / cats::kSparseCols;
  // about one block per compute unit; one group once the column tiles alone
  // fill most of the chip
  L.NG = (cats::kFusedBlocks + L.CT / 2) / L.CT;
  if (L.NG < 1) L.NG = 1;
  if (L.NG > d) L.NG = d;
  if (L.NG > cats::kFusedBlocks) L.NG = cats::kFusedBlocks;
  size_t o = radix_bytes();
  L.partial = o;
  o = round_up(o + (size_t)L.NG * B * n * sizeof(float), kAlign);
  L.tickets = o;
  o = round_up(o + (size_t)L.CT * sizeof(unsigned long long), kAlign);
  L.seg_j = o;
  o = round_up(o + (size_t)d * sizeof(int32_t), kAlign);
  L.seg_mask = o;
  o = round_up(o + (size_t)d * sizeof(uint32_t), kAlign);
  L.seg_v = o;
  o = round_up(o + (size_t)B * d * sizeof(float), kAlign);
  L.seg_h = o;
  o = round_up(o + (size_t)B * d * sizeof(float), kAlign);
  L.seg_cnt = o;
  o = round_up(o + (size_t)cats::kFusedBlocks * sizeof(int32_t), kAlign);
  L.end = o;
  return L;
}

// Tags of successive ticketed calls (sparse input, the top-k select; never
// 0), so a ticket word left by any earlier call is recognised as stale.  The
// sequence starts at a random point of the 32-bit range, not at 1: a
// workspace shared between entry points can leave data in a ticket word,
// and data is full of small integers (indices, counts), which a counter
// starting at 1 would meet within its first thousands of calls.
uint32_t epoch_start() {
  uint32_t s = 0x9e3779b9u;
  try {
    std::random_device rd;
    s ^= rd();
  } catch (...) {
  }
  s ^= (uint32_t)std::chrono::steady_clock::now().time_since_epoch().count();
  s ^= (uint32_t)(reinterpret_cast<uintptr_t>(&s) >> 4);
  return s;
}
std::atomic<uint32_t> g_epoch{epoch_start()};
uint32_t next_epoch() {
  uint32_t e;
  do {
    e = g_epoch.fetch_add(1u, std::memory_order_relaxed) + 1u;
  } while (e == 0u);
  return e;
}

bool gemv_shape_ok(int d, int n) {
  return d > 0 && d <= CATS_MAX_M && n > 0 && n % 8 == 0 && (uint64_t)d * n * 2 <= CATS_MAX_MATRIX_BYTES;
}
}  // namespace

size_t cats_sparse_input_workspace_bytes(int32_t d, int32_t n, int32_t max_batch) {
  if (!gemv_shape_ok(d, n) || max_batch < 1 || max_batch > CATS_MAX_BATCH) return 0;
  return gemv_layout(d, n, max_batch).end;
}

cats_status cats_sparse_input_gemv(const void* w, int32_t d, int32_t n, int32_t wdtype, const float* x,
                                   int32_t B, float t, const float* residual, float* y,
                                   const cats_forward_aux* aux, void* ws, size_t ws_bytes, void* stream) {
  if (!w || !x || !y) return fail(CATS_ERR_NULL, "w, x or y is NULL");
  if (wdtype != CATS_BF16 && wdtype != CATS_F32) return fail(CATS_ERR_DTYPE, "unknown weight dtype %d", (int)wdtype);
  if (wdtype != CATS_BF16) return fail(CATS_ERR_UNIMPLEMENTED, "the sparse-input product takes bf16 weights");
  if (!gemv_shape_ok(d, n))
    return fail(CATS_ERR_SHAPE, "d=%d must be in [1, %d], n=%d a positive multiple of 8, d*n*2 at most %llu bytes",
                (int)d, CATS_MAX_M, (int)n, (unsigned long long)CATS_MAX_MATRIX_BYTES);
  if (B < 1 || B > CATS_MAX_BATCH) return fail(CATS_ERR_SHAPE, "B=%d outside [1, %d]", (int)B, CATS_MAX_BATCH);
  if (!aligned(w, 16) || !aligned(x, 4) || !aligned(y, 16) || (residual && !aligned(residual, 16)))
    return fail(CATS_ERR_ALIGN, "w, y and residual must be 16-byte aligned, x 4-byte aligned");
  if (std::isnan(t) || t < 0.f) return fail(CATS_ERR_RANGE, "t must be >= 0 (got %g)", (double)t);
  const bool want_aux = aux && (aux->active_idx || aux->active_cnt || aux->active_v || aux->active_h);
  if (want_aux && ((aux->active_idx && !aligned(aux->active_idx, 4)) ||
                   (aux->active_cnt && !aligned(aux->active_cnt, 4)) ||
                   (aux->active_v && !aligned(aux->active_v, 4)) ||
                   (aux->active_h && !aligned(aux->active_h, 4))))
    return fail(CATS_ERR_ALIGN, "aux outputs must be 4-byte aligned");
  const GemvLayout lay = gemv_layout(d, n, B);
  cats_status st = check_ws(ws, ws_bytes, lay.end);
  if (st != CATS_OK) return st;
  char* wsp = static_cast<char*>(ws);
  const hipStream_t s = static_cast<hipStream_t>(stream);

  cats::SparseInputArgs sa;
  sa.w = w;
  sa.x = x;
  sa.residual = residual;
  sa.y = y;
  sa.B = B;
  sa.d = d;
  sa.n = n;
  sa.t = t;
  sa.NG = lay.NG;
  sa.CT = lay.CT;
  sa.partial = reinterpret_cast<float*>(wsp + lay.partial);
  sa.tickets = reinterpret_cast<unsigned long long*>(wsp + lay.tickets);
  sa.epoch = next_epoch();
  sa.aux = want_aux ? 1 : 0;
  sa.seg_j = reinterpret_cast<int*>(wsp + lay.seg_j);
  sa.seg_mask = reinterpret_cast<uint32_t*>(wsp + lay.seg_mask);
  sa.seg_v = reinterpret_cast<float*>(wsp + lay.seg_v);
  sa.seg_h = reinterpret_cast<float*>(wsp + lay.seg_h);
  sa.seg_cnt = reinterpret_cast<int*>(wsp + lay.seg_cnt);
  hipError_t e = cats::launch_sparse_input(sa, s);
  if (e != hipSuccess) return hip_fail(e, "sparse-input product launch");
  if (want_aux) {
    // the per-row active lists from the groups' segments (y is written)
    cats::ReduceArgs ra;
    ra.partial = nullptr;
    ra.G = lay.NG;
    ra.Gseg = lay.NG;
    ra.sum_y = 0;
    ra.B = B;
    ra.d = n;
    ra.m = d;
    ra.residual = nullptr;
    ra.y = nullptr;
    ra.aux = 1;
    ra.seg_j = sa.seg_j;
    ra.seg_mask = sa.seg_mask;
    ra.seg_v = sa.seg_v;
    ra.seg_h = sa.seg_h;
    ra.seg_cnt = sa.seg_cnt;
    ra.active_idx = aux->active_idx;
    ra.active_cnt = aux->active_cnt;
    ra.active_v = aux->active_v;
    ra.active_h = aux->active_h;
    e = cats::launch_reduce(ra, s);
    if (e != hipSuccess) return hip_fail(e, "active-list launch");
  }
  return sync_check(stream, "cats_sparse_input_gemv");
}

namespace {
// Workspace of cats_calibrate_stack: the general region (calibration
// activations, or the forward's partials while vectors are propagated),
// then the propagated vectors X and their RMSNorm XN, [N x d] each.
size_t stack_calib_general(int d, int max_m, int N) {
  const size_t cal = calib_bytes((int64_t)N * max_m);
  const size_t fwd = fwd_layout(d, max_m, CATS_MAX_BATCH).end + stack_rows_bytes(d, CATS_MAX_BATCH);
  return cal > fwd ? cal : fwd;
}
}  // namespace

size_t cats_calibrate_stack_workspace_bytes(int32_t d, int32_t max_m, int32_t N) {
  if (d <= 0 || d % 8 != 0 || d > CATS_MAX_D_BF16 || max_m <= 0 || max_m > CATS_MAX_M || N <= 0 ||
      N > 4 * 1024 * 1024 || (int64_t)N * max_m > (int64_t)0xffffffffll)
    return 0;
  return stack_calib_general(d, max_m, N) + 2 * round_up((size_t)N * d * sizeof(float), kAlign);
}

cats_status cats_calibrate_stack(const cats_layer* layers, int32_t L, const float* calib_x, int32_t N,
                                 double sparsity, float eps, void* ws, size_t ws_bytes, void* stream,
                                 float* t_out) {
  if (!layers || !calib_x || !t_out) return fail(CATS_ERR_NULL, "layers, calib_x or t_out is NULL");
  if (L < 1 || L > CATS_MAX_LAYERS) return fail(CATS_ERR_SHAPE, "L=%d outside [1, %d]", (int)L, CATS_MAX_LAYERS);
  if (N <= 0 || N > 4 * 1024 * 1024) return fail(CATS_ERR_SHAPE, "N=%d out of range", (int)N);
  if (!aligned(calib_x, 16)) return fail(CATS_ERR_ALIGN, "calib_x must be 16-byte aligned");
  if (!std::isfinite(sparsity) || sparsity < 0.0 || sparsity > 1.0)
    return fail(CATS_ERR_RANGE, "sparsity must be in [0, 1]");
  if (!std::isfinite(eps) || eps < 0.f) return fail(CATS_ERR_RANGE, "eps must be finite and >= 0");
  const int d = layers[0].d;
  int max_m = 0;
  for (int l = 0; l < L; ++l) {
    cats_status st = check_layer(&layers[l]);
    if (st != CATS_OK) return fail(st, "layer %d: %s", l, g_last_error.c_str());
    if (layers[l].d != d) return fail(CATS_ERR_SHAPE, "layer %d has d=%d, layer 0 has d=%d", l, (int)layers[l].d, d);
    if (layers[l].m > max_m) max_m = layers[l].m;
  }
  if ((int64_t)N * max_m > (int64_t)0xffffffffll) return fail(CATS_ERR_SHAPE, "N*m too large");
  if (sparsity == 0.0) {
    for (int l = 0; l < L; ++l) t_out[l] = 0.f;
    return CATS_OK;
  }
  const size_t general = stack_calib_general(d, max_m, N);
  const size_t rows = round_up((size_t)N * d * sizeof(float), kAlign);
  cats_status st = check_ws(ws, ws_bytes, general + 2 * rows);
  if (st != CATS_OK) return st;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  float* X = reinterpret_cast<float*>(static_cast<char*>(ws) + general);
  float* XN = reinterpret_cast<float*>(static_cast<char*>(ws) + general + rows);
  float* acts = reinterpret_cast<float*>(static_cast<char*>(ws) + radix_bytes());
  hipError_t e = hipMemcpyAsync(X, calib_x, (size_t)N * d * sizeof(float), hipMemcpyDeviceToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "calibration vector copy");
  for (int l = 0; l < L; ++l) {
    const cats_layer* ly = &layers[l];
    // what block l sees: the RMSNorm of the densely propagated vectors
    e = cats::launch_rmsnorm(X, XN, N, d, eps, s);
    if (e != hipSuccess) return hip_fail(e, "rmsnorm launch");
    e = cats::launch_calib_acts(ly->wdtype == CATS_BF16, XN, ly->w_gate_t, N, d, ly->m, acts, s);
    if (e != hipSuccess) return hip_fail(e, "calibration activations launch");
    st = select_threshold(acts, (int64_t)N * ly->m, sparsity, ws, s, &t_out[l]);
    if (st != CATS_OK) return st;
    if (l == L - 1) break;
    // X <- X + dense MLP_l(XN), CATS_MAX_BATCH rows per call
    for (int r0 = 0; r0 < N; r0 += CATS_MAX_BATCH) {
      const int nb = (N - r0) < CATS_MAX_BATCH ? (N - r0) : CATS_MAX_BATCH;
      float* xr = X + (size_t)r0 * d;
      st = run_mlp(ly, XN + (size_t)r0 * d, nb, 0.f, true, xr, xr, nullptr, ws, general, stream);
      if (st != CATS_OK) return fail(st, "layer %d propagation: %s", l, g_last_error.c_str());
    }
  }
  return CATS_OK;
}

// Top-k workspace: the forward's, then v [B x m], the cutoffs [B] and the
// gate blocks' arrival count of the in-kernel select (one 64-bit word).
size_t cats_topk_workspace_bytes(int32_t d, int32_t m, int32_t max_batch) {
  const size_t base = round_up(cats_workspace_bytes(d, m, max_batch, 0), kAlign);
  if (base == 0) return 0;
  return base + round_up((size_t)max_batch * m * sizeof(float), kAlign) +
         round_up((size_t)max_batch * sizeof(float), kAlign) + kAlign;
}

cats_status cats_mlp_forward_topk(const cats_layer* layer, const float* x, int32_t B, double sparsity,
                                  const float* residual, float* y, const cats_forward_aux* aux, void* ws,
                                  size_t ws_bytes, void* stream, float* t_out) {
  cats_status st = check_layer(layer);
  if (st != CATS_OK) return st;
  if (!x || !y) return fail(CATS_ERR_NULL, "x or y is NULL");
  if (B < 1 || B > CATS_MAX_BATCH) return fail(CATS_ERR_SHAPE, "B=%d outside [1, %d]", (int)B, CATS_MAX_BATCH);
  if (!std::isfinite(sparsity) || sparsity < 0.0 || sparsity > 1.0)
    return fail(CATS_ERR_RANGE, "sparsity must be in [0, 1]");
  if (!aligned(x, 16) || !aligned(y, 16) || (residual && !aligned(residual, 16)))
    return fail(CATS_ERR_ALIGN, "x, y and residual must be 16-byte aligned");
  if (t_out && !aligned(t_out, 4)) return fail(CATS_ERR_ALIGN, "t_out must be 4-byte aligned");
  if (aux && ((aux->active_idx && !aligned(aux->active_idx, 4)) || (aux->active_cnt && !aligned(aux->active_cnt, 4)) ||
              (aux->active_v && !aligned(aux->active_v, 4)) || (aux->active_h && !aligned(aux->active_h, 4))))
    return fail(CATS_ERR_ALIGN, "aux outputs must be 4-byte aligned");
  const int d = layer->d, m = layer->m;
  const int bf16 = layer->wdtype == CATS_BF16;
  const size_t base = round_up(cats_workspace_bytes(d, m, B, 0), kAlign);
  st = check_ws(ws, ws_bytes, cats_topk_workspace_bytes(d, m, B));
  if (st != CATS_OK) return st;
  float* vbuf = reinterpret_cast<float*>(static_cast<char*>(ws) + base);
  float* tbuf = reinterpret_cast<float*>(static_cast<char*>(ws) + base + round_up((size_t)B * m * sizeof(float), kAlign));
  unsigned long long* ticket = reinterpret_cast<unsigned long long*>(
      reinterpret_cast<char*>(tbuf) + round_up((size_t)B * sizeof(float), kAlign));
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int nch = cats::fused_nch(bf16, d);
  const int bt_max = cats::fused_bt_max(bf16, nch);
  const int G = cats::fused_grid(m);
  const int64_t rank = cutoff_rank(m, sparsity);
  // One row of up to kGateSelMaxM neurons: the gate kernel's last block
  // selects the cutoff itself (no select launch).
  const bool sel_in_gate = B == 1 && m <= cats::kGateSelMaxM;
  if (sel_in_gate) {
    cats::GateVArgs ga{};
    ga.wg = layer->w_gate_t;
    ga.x = x;
    ga.B = 1;
    ga.d = d;
    ga.m = m;
    ga.v = vbuf;
    ga.rank = (int)rank;
    ga.t_out = tbuf;
    ga.ticket = ticket;
    ga.epoch = next_epoch();
    hipError_t e = cats::launch_gate_v_select(bf16, nch, ga, G, s);
    if (e != hipSuccess) return hip_fail(e, "gate activation and cutoff launch");
  } else {
    for (int b0 = 0; b0 < B; b0 += bt_max) {
      const int bp = (B - b0) < bt_max ? (B - b0) : bt_max;
      cats::GateVArgs ga{};
      ga.wg = layer->w_gate_t;
      ga.x = x + (size_t)b0 * d;
      ga.B = bp;
      ga.d = d;
      ga.m = m;
      ga.v = vbuf + (size_t)b0 * m;
      hipError_t e = cats::launch_gate_v(bf16, nch, batch_tile(bp), false, ga, G, s);
      if (e != hipSuccess) return hip_fail(e, "gate activation launch");
    }
  }
  hipError_t e = hipSuccess;
  if (!sel_in_gate) {
    e = cats::launch_row_select(vbuf, B, m, rank, tbuf, s);
    if (e != hipSuccess) return hip_fail(e, "per-row cutoff launch");
  }
  st = run_mlp(layer, x, B, 0.f, false, residual, y, aux, ws, base, stream, false, 0.f, vbuf, tbuf);
  if (st != CATS_OK) return st;
  if (t_out) {
    e = hipMemcpyAsync(t_out, tbuf, (size_t)B * sizeof(float), hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "cutoff copy");
  }
  return sync_check(stream, "cats_mlp_forward_topk");
}

size_t cats_unfused_workspace_bytes(int32_t d, int32_t m, int32_t max_batch) {
  const size_t base = round_up(cats_workspace_bytes(d, m, max_batch, 0), kAlign);
  if (base == 0) return 0;
  return base + 2 * round_up((size_t)max_batch * m * sizeof(float), kAlign);
}

cats_status cats_mlp_forward_unfused(const cats_layer* layer, const float* x, int32_t B, float t, int32_t mode,
                                     const float* residual, float* y, void* ws, size_t ws_bytes, void* stream) {
  cats_status st = check_layer(layer);
  if (st != CATS_OK) return st;
  if (!x || !y) return fail(CATS_ERR_NULL, "x or y is NULL");
  if (B < 1 || B > CATS_MAX_BATCH) return fail(CATS_ERR_SHAPE, "B=%d outside [1, %d]", (int)B, CATS_MAX_BATCH);
  if (mode != CATS_UNFUSED_MASK && mode != CATS_UNFUSED_INDEX) return fail(CATS_ERR_RANGE, "unknown mode %d", (int)mode);
  if (std::isnan(t) || t < 0.f) return fail(CATS_ERR_RANGE, "t must be >= 0 (got %g)", (double)t);
  if (!aligned(x, 16) || !aligned(y, 16) || (residual && !aligned(residual, 16)))
    return fail(CATS_ERR_ALIGN, "x, y and residual must be 16-byte aligned");
  const int d = layer->d, m = layer->m;
  const int bf16 = layer->wdtype == CATS_BF16;
  st = check_ws(ws, ws_bytes, cats_unfused_workspace_bytes(d, m, B));
  if (st != CATS_OK) return st;
  const bool index = mode == CATS_UNFUSED_INDEX;
  const size_t base = round_up(cats_workspace_bytes(d, m, B, 0), kAlign);
  char* w = static_cast<char*>(ws);
  const FwdLayout lay = fwd_layout(d, m, B);
  float* vbuf = reinterpret_cast<float*>(w + base);
  float* hbuf = reinterpret_cast<float*>(w + base + round_up((size_t)B * m * sizeof(float), kAlign));
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int nch = cats::fused_nch(bf16, d);
  const int bt_max = cats::fused_bt_max(bf16, nch);
  const int G = cats::fused_grid(m);
  for (int b0 = 0; b0 < B; b0 += bt_max) {
    const int bp = (B - b0) < bt_max ? (B - b0) : bt_max;
    const int bt = batch_tile(bp);
    cats::GateVArgs ga{};
    ga.wg = layer->w_gate_t;
    ga.x = x + (size_t)b0 * d;
    ga.B = bp;
    ga.d = d;
    ga.m = m;
    ga.v = vbuf;
    ga.t = t;
    ga.seg_j = reinterpret_cast<int*>(w + lay.seg_j);
    ga.seg_mask = reinterpret_cast<uint32_t*>(w + lay.seg_mask);
    ga.seg_cnt = reinterpret_cast<int*>(w + lay.seg_cnt);
    hipError_t e = cats::launch_gate_v(bf16, nch, bt, index, ga, G, s);
    if (e != hipSuccess) return hip_fail(e, "gate launch");
    cats::UnfusedArgs ua{};
    ua.wu = layer->w_up_t;
    ua.wd = layer->w_down;
    ua.x = ga.x;
    ua.v = vbuf;
    ua.t = t;
    ua.B = bp;
    ua.d = d;
    ua.m = m;
    ua.seg_j = ga.seg_j;
    ua.seg_cnt = ga.seg_cnt;
    ua.h = hbuf;
    ua.partial = reinterpret_cast<float*>(w + lay.partial);
    e = cats::launch_unfused_up(bf16, nch, bt, index, ua, G, s);
    if (e != hipSuccess) return hip_fail(e, "up-projection launch");
    e = cats::launch_unfused_down(bf16, nch, bt, index, ua, G, s);
    if (e != hipSuccess) return hip_fail(e, "down-projection launch");
    cats::ReduceArgs ra{};
    ra.partial = ua.partial;
    ra.G = G;
    ra.Gseg = G;
    ra.sum_y = 1;
    ra.B = bp;
    ra.d = d;
    ra.m = m;
    ra.residual = residual ? residual + (size_t)b0 * d : nullptr;
    ra.y = y + (size_t)b0 * d;
    ra.aux = 0;
    e = cats::launch_reduce(ra, s);
    if (e != hipSuccess) return hip_fail(e, "reduce launch");
  }
  return sync_check(stream, "cats_mlp_forward_unfused");
}

cats_status cats_rmsnorm(const float* x, float* xn, int32_t B, int32_t d, float eps, void* stream) {
  if (!x || !xn) return fail(CATS_ERR_NULL, "x or xn is NULL");
  if (B < 1 || B > 65535 || d < 1) return fail(CATS_ERR_SHAPE, "B=%d, d=%d out of range", (int)B, (int)d);
  if (std::isnan(eps) || eps < 0.f) return fail(CATS_ERR_RANGE, "eps must be >= 0");
  if (!aligned(x, 4) || !aligned(xn, 4)) return fail(CATS_ERR_ALIGN, "x and xn must be 4-byte aligned");
  hipError_t e = cats::launch_rmsnorm(x, xn, B, d, eps, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "rmsnorm launch");
  return sync_check(stream, "cats_rmsnorm");
}

cats_status cats_stream_read(const void* buf, size_t bytes, int32_t blocks, int32_t inflight, int32_t runs,
                             uint32_t* sink, void* stream) {
  if (!buf || !sink) return fail(CATS_ERR_NULL, "buf or sink is NULL");
  if (bytes == 0 || bytes % 16 != 0 || bytes > cats::kStreamReadMaxBytes)
    return fail(CATS_ERR_SHAPE, "bytes=%zu must be a positive multiple of 16 of at most %llu", bytes,
                (unsigned long long)cats::kStreamReadMaxBytes);
  if (blocks < 1 || blocks > 65536) return fail(CATS_ERR_SHAPE, "blocks=%d outside [1, 65536]", (int)blocks);
  if (inflight != 4 && inflight != 8 && inflight != 16)
    return fail(CATS_ERR_RANGE, "inflight=%d must be 4, 8 or 16", (int)inflight);
  if (runs != 0 && runs != 1) return fail(CATS_ERR_RANGE, "runs=%d must be 0 or 1", (int)runs);
  if (!aligned(buf, 16) || !aligned(sink, 4)) return fail(CATS_ERR_ALIGN, "buf must be 16-byte aligned, sink 4");
  hipError_t e = cats::launch_stream_read(buf, (uint32_t)bytes, blocks, inflight, runs != 0, sink,
                                          static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "stream read launch");
  return sync_check(stream, "cats_stream_read");
}

cats_status cats_timer_enable(int32_t on) {
  TimerState& T = timer_state();
  std::lock_guard<std::mutex> lk(T.mu);
  T.on = on != 0;
  return CATS_OK;
}

cats_status cats_timer_reset(void) {
  TimerState& T = timer_state();
  std::lock_guard<std::mutex> lk(T.mu);
  hipError_t e = T.pending.empty() ? hipSuccess : timer_flush_locked(T);
  for (size_t i = 0; i < T.names.size(); ++i) {
    T.launches[i] = 0;
    T.total_ms[i] = 0.0;
  }
  if (e != hipSuccess) return hip_fail(e, "timer flush");
  return CATS_OK;
}

int32_t cats_timer_count(void) {
  TimerState& T = timer_state();
  std::lock_guard<std::mutex> lk(T.mu);
  return (int32_t)T.names.size();
}

cats_status cats_timer_get(int32_t i, const char** name, int64_t* launches, double* total_ms) {
  TimerState& T = timer_state();
  std::lock_guard<std::mutex> lk(T.mu);
  if (i < 0 || i >= (int32_t)T.names.size()) return fail(CATS_ERR_RANGE, "timer index %d out of range", (int)i);
  hipError_t e = T.pending.empty() ? hipSuccess : timer_flush_locked(T);
  if (e != hipSuccess) return hip_fail(e, "timer flush");
  if (name) *name = T.names[i].c_str();
  if (launches) *launches = T.launches[i];
  if (total_ms) *total_ms = T.total_ms[i];
  return CATS_OK;
}

}  // extern "C"
