// Host side of the C ABI declared in include/dominotree.h: argument checks,
// plan creation (weight packing), workspace layout and launch sequencing.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <new>
#include <string>

#include "dt_internal.h"
#include "dt_select.h"

namespace {

thread_local std::string g_last_error;

dt_status fail(dt_status s, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
dt_status fail(dt_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

dt_status hip_fail(hipError_t e, const char *what) {
  return fail(DT_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

bool valid_dtype(int d) { return d == DT_F32 || d == DT_BF16; }
size_t dsize(int d) { return d == DT_BF16 ? 2 : 4; }

int ecap_for(const dt_plan *p) { return p->L * p->B + dt::kChunkNodes; }

// ---- scratch of the allocation-free entry point (dt_build_tree_noalloc) ----
constexpr size_t kScratchBytes = (size_t)32 << 20;  // 32 MiB per device
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];  // the array's device address on each device (null: not yet)

}  // namespace

// The workspace of dt_build_tree_noalloc: one array per device, alive until the
// process ends.  Its name is a host-side stand-in; kernels get the address that
// hipGetSymbolAddress returns for the current device (scratch_address).
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

// The scratch array's address on the current device, resolved once per device.
hipError_t scratch_address(int dev, void **ptr) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *q = nullptr;
    const hipError_t e = hipGetSymbolAddress(&q, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = q;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

namespace dt {

// Lay out the workspace of one dt_build_tree call; base == nullptr only sizes it.
Workspace carve(const dt_plan *p, int batch, char *base) {
  Workspace ws{};
  const int rows = batch * p->L;
  const ScanGeom g = scan_geom(rows, p->V, p->M);
  size_t o = base ? carve_scan(base, g, &ws) : scan_bytes(g);
  auto at = [&](size_t bytes) {
    float *ptr = base ? reinterpret_cast<float *>(base + o) : nullptr;
    o += align_up(bytes, 256);
    return ptr;
  };
  ws.ecap = ecap_for(p);
  ws.states = at((size_t)batch * ws.ecap * p->d_h * sizeof(float));
  ws.part = at(expand_part_bytes(p, batch));
  // per tree: barrier counters; then the member-slot counters of the launch
  // (two sets: a call makes up to two expansion launches)
  ws.bar = reinterpret_cast<int32_t *>(at((size_t)2 * (batch + kSlotRows) * kBarStride * sizeof(int32_t)));
  ws.menus = p->scorer == DT_SCORER_STATIC
                 ? at((size_t)batch * p->L * ((p->M + 63) / 64 * 64) * sizeof(float))
                 : nullptr;
  ws.bytes = o;
  return ws;
}

}  // namespace dt

extern "C" {

int dt_abi_version(void) { return DT_ABI_VERSION; }

const char *dt_status_string(int s) {
  switch (s) {
    case DT_OK: return "ok";
    case DT_ERR_NULL: return "a required pointer is NULL";
    case DT_ERR_SHAPE: return "a size is out of range or inconsistent";
    case DT_ERR_DTYPE: return "unknown dtype";
    case DT_ERR_UNSUPPORTED: return "outside the supported envelope";
    case DT_ERR_WORKSPACE: return "workspace missing or too small";
    case DT_ERR_ALIGN: return "misaligned pointer";
    case DT_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char *dt_last_error(void) { return g_last_error.c_str(); }

// the options (NULL: defaults) checked into *o
static dt_status check_options(const dt_options *opts, dt_options *o) {
  *o = dt_options{0, DT_NORM_TAIL, 0, 0, 0, 0};
  if (opts) *o = *opts;
  if (o->max_children < 0) return fail(DT_ERR_SHAPE, "max_children must be >= 0");
  if (o->frontier_width < 0 || o->debug_spin_limit < 0)
    return fail(DT_ERR_SHAPE, "frontier_width and debug_spin_limit must be >= 0");
  if (o->norm_mode != DT_NORM_TAIL && o->norm_mode != DT_NORM_SLICE)
    return fail(DT_ERR_UNSUPPORTED, "norm_mode must be DT_NORM_TAIL or DT_NORM_SLICE");
  if (o->scorer != DT_SCORER_COND && o->scorer != DT_SCORER_MARG && o->scorer != DT_SCORER_STATIC)
    return fail(DT_ERR_UNSUPPORTED, "scorer must be DT_SCORER_COND, DT_SCORER_MARG or DT_SCORER_STATIC");
  return DT_OK;
}

// drop one reference; the last one frees the tables
static void model_release(dt_model *m) {
  if (!m || m->refs.fetch_sub(1) != 1) return;
  if (m->wfold) (void)hipFree(m->wfold);
  if (m->b_ih) (void)hipFree(m->b_ih);
  if (m->b_hh) (void)hipFree(m->b_hh);
  if (m->b_c) (void)hipFree(m->b_c);
  if (m->whh_t) (void)hipFree(m->whh_t);
  if (m->whh_rm) (void)hipFree(m->whh_rm);
  if (m->P_all) (void)hipFree(m->P_all);
  if (m->U_all) (void)hipFree(m->U_all);
  if (m->c_all) (void)hipFree(m->c_all);
  delete m;
}

dt_status dt_model_create(dt_model **model, const void *emb, int V, int d_e, const dt_gru *gru,
                          const dt_head *head, int weights_dtype) {
  if (!model) return fail(DT_ERR_NULL, "model out-pointer is NULL");
  *model = nullptr;
  if (!emb || !gru || !head) return fail(DT_ERR_NULL, "emb, gru and head are required");
  if (!gru->w_ih || !gru->w_hh || !head->w) return fail(DT_ERR_NULL, "w_ih, w_hh and head.w are required");
  if (!valid_dtype(weights_dtype)) return fail(DT_ERR_DTYPE, "dtype codes must be DT_F32 or DT_BF16");
  if (V < 1 || d_e < 1) return fail(DT_ERR_SHAPE, "sizes must be positive (V=%d d_e=%d)", V, d_e);
  if (gru->d_in != d_e) return fail(DT_ERR_SHAPE, "gru.d_in (%d) must equal d_e (%d)", gru->d_in, d_e);
  const int d_h = gru->d_h;
  if (d_e > dt::kMaxDe || d_h < 32 || d_h > dt::kMaxDh || d_h % 32 != 0)
    return fail(DT_ERR_UNSUPPORTED, "outside the envelope (d_e<=8192, 32<=d_h<=1024, d_h%%32==0)");
  const size_t ws = dsize(weights_dtype);
  if (!aligned(emb, 16) || !aligned(gru->w_ih, ws) || !aligned(gru->w_hh, ws) ||
      !aligned(head->w, ws) || (gru->b_ih && !aligned(gru->b_ih, ws)) ||
      (gru->b_hh && !aligned(gru->b_hh, ws)) || (head->b && !aligned(head->b, ws)))
    return fail(DT_ERR_ALIGN, "emb must be 16-byte aligned, weights naturally aligned");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "device query");
  dt_model *m = new (std::nothrow) dt_model();
  if (!m) return fail(DT_ERR_HIP, "host allocation failed");
  m->refs.store(1);
  m->V = V;
  m->d_e = d_e;
  m->d_h = d_h;
  m->wdt = weights_dtype;
  m->emb = emb;
  m->nf = 4 * d_h;
  m->nf_pad = (m->nf + dt::kFoldBN - 1) / dt::kFoldBN * dt::kFoldBN;
  m->has_bc = head->b != nullptr;
  m->device = dev;
  e = hipMalloc(&m->wfold, (size_t)m->nf_pad * d_e * ws);
  if (e == hipSuccess) e = hipMalloc(&m->b_ih, sizeof(float) * 3 * d_h);
  if (e == hipSuccess) e = hipMalloc(&m->b_hh, sizeof(float) * 3 * d_h);
  if (e == hipSuccess) e = hipMalloc(&m->b_c, sizeof(float) * d_e);
  if (e == hipSuccess) e = hipMalloc(&m->whh_t, (size_t)3 * d_h * d_h * ws);
  if (e == hipSuccess) e = hipMalloc(&m->whh_rm, (size_t)3 * d_h * d_h * ws);
  if (e == hipSuccess)
    e = hipMemcpyAsync(m->whh_rm, gru->w_hh, (size_t)3 * d_h * d_h * ws, hipMemcpyDeviceToDevice,
                       nullptr);
  if (e == hipSuccess) e = hipMalloc(&m->P_all, (size_t)V * 3 * d_h * sizeof(float));
  if (e == hipSuccess) e = hipMalloc(&m->U_all, (size_t)V * d_h * sizeof(float));
  if (e == hipSuccess) e = hipMalloc(&m->c_all, (size_t)V * sizeof(float));
  if (e == hipSuccess) e = dt::pack_weights(m, gru, head, nullptr);
  if (e == hipSuccess) e = dt::fold_vocab(m, nullptr);
  if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
  if (e == hipSuccess) {
    e = hipFree(m->wfold);
    m->wfold = nullptr;
  }
  m->emb = nullptr;  // (only read while the tables are built)
  if (e != hipSuccess) {
    dt_status st = hip_fail(e, "model creation");
    model_release(m);
    return st;
  }
  *model = m;
  return DT_OK;
}

void dt_model_destroy(dt_model *model) { model_release(model); }

dt_status dt_plan_create_from_model(dt_plan **plan, dt_model *model, int L, int M, int B,
                                    int logits_dtype, int max_batch, const dt_options *opts) {
  if (!plan) return fail(DT_ERR_NULL, "plan out-pointer is NULL");
  *plan = nullptr;
  if (!model) return fail(DT_ERR_NULL, "model is required");
  if (!valid_dtype(logits_dtype)) return fail(DT_ERR_DTYPE, "dtype codes must be DT_F32 or DT_BF16");
  const int V = model->V, d_h = model->d_h;
  if (L < 1 || M < 1 || B < 1 || max_batch < 1)
    return fail(DT_ERR_SHAPE, "sizes must be positive (L=%d M=%d B=%d max_batch=%d)", L, M, B, max_batch);
  if (M > V) return fail(DT_ERR_SHAPE, "M (%d) exceeds V (%d)", M, V);
  if (M > dt::kMaxM || B > dt::kMaxB || L > dt::kMaxL)
    return fail(DT_ERR_UNSUPPORTED, "outside the envelope (M<=256, B<=256, L<=64)");
  dt_options o;
  const dt_status ost = check_options(opts, &o);
  if (ost != DT_OK) return ost;
  int dev = 0, ncu = 0, maxlds = 0, nxcd = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&nxcd, hipDeviceAttributeNumberOfXccs, dev);
  if (e == hipSuccess)
    e = hipDeviceGetAttribute(&maxlds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return hip_fail(e, "device query");
  if (dev != model->device)
    return fail(DT_ERR_SHAPE, "the model lives on device %d, the current device is %d", model->device, dev);
  if (nxcd < 1 || nxcd > dt::kMaxXcd)
    return fail(DT_ERR_UNSUPPORTED, "device reports %d XCDs; 1 to %d are supported", nxcd, dt::kMaxXcd);
  if (dt::merge_lds_bytes(dt::scan_geom(1, V, M)) > (size_t)dt::kMergeLdsMax)
    return fail(DT_ERR_UNSUPPORTED, "the row merge of V and M needs %zu bytes of LDS, more than %d",
                dt::merge_lds_bytes(dt::scan_geom(1, V, M)), dt::kMergeLdsMax);
  // the expansion's LDS at the group size of every batch in [1, max_batch]
  // (the group shrinks until its layout fits; only one member per tree can
  // still be too large)
  size_t lds_need = 0;
  for (int b = 1; b <= max_batch; ++b) {
    const int nb = dt::scan_geom(b * L, V, M).nchunks;
    const int G = dt::expand_group_size(d_h, ncu, nxcd, b, M, L, nb, (size_t)maxlds);
    const size_t need = dt::expand_lds_bytes(d_h, G, M, nb, L);
    lds_need = need > lds_need ? need : lds_need;
  }
  if (lds_need > (size_t)maxlds)
    return fail(DT_ERR_UNSUPPORTED,
                "expansion needs %zu bytes of LDS (d_h=%d, M=%d, max_batch=%d), device has %d",
                lds_need, d_h, M, max_batch, maxlds);
  void *scratch_ptr = nullptr;
  e = scratch_address(dev, &scratch_ptr);  // once per device: dt_build_tree_noalloc's workspace
  if (e != hipSuccess) return hip_fail(e, "scratch address");

  dt_plan *p = new (std::nothrow) dt_plan();
  if (!p) return fail(DT_ERR_HIP, "host allocation failed");
  model->refs.fetch_add(1);
  p->model = model;
  p->V = V;
  p->d_e = model->d_e;
  p->d_h = d_h;
  p->wdt = model->wdt;
  p->P_all = model->P_all;
  p->U_all = model->U_all;
  p->c_all = model->c_all;
  p->b_ih = model->b_ih;
  p->b_hh = model->b_hh;
  p->whh_t = model->whh_t;
  p->whh_rm = model->whh_rm;
  p->L = L;
  p->M = M;
  p->B = B;
  int k = o.max_children > 0 ? o.max_children : (M < B ? M : B);
  if (k > M) k = M;
  if (k > B) k = B;  // a child ranked B or lower among its siblings can never be popped
  p->k = k;
  p->norm_mode = o.norm_mode;
  p->scorer = o.scorer;
  p->pos_offset = o.pos_offset;
  p->ldt = logits_dtype;
  p->max_batch = max_batch;
  p->num_cus = ncu;
  p->num_xcd = nxcd;
  p->max_lds = (size_t)maxlds;
  p->frontier_w = o.frontier_width;
  p->spin_limit = o.debug_spin_limit;
  p->device = dev;
  *plan = p;
  return DT_OK;
}

dt_status dt_plan_create(dt_plan **plan, const void *emb, int V, int d_e, const dt_gru *gru,
                         const dt_head *head, int weights_dtype, int L, int M, int B,
                         int logits_dtype, int max_batch, const dt_options *opts) {
  if (!plan) return fail(DT_ERR_NULL, "plan out-pointer is NULL");
  *plan = nullptr;
  // the plain shape checks come before the (large) tables are built
  if (!valid_dtype(logits_dtype)) return fail(DT_ERR_DTYPE, "dtype codes must be DT_F32 or DT_BF16");
  if (L < 1 || M < 1 || B < 1 || max_batch < 1)
    return fail(DT_ERR_SHAPE, "sizes must be positive (L=%d M=%d B=%d max_batch=%d)", L, M, B, max_batch);
  if (V >= 1 && M > V) return fail(DT_ERR_SHAPE, "M (%d) exceeds V (%d)", M, V);
  if (M > dt::kMaxM || B > dt::kMaxB || L > dt::kMaxL)
    return fail(DT_ERR_UNSUPPORTED, "outside the envelope (M<=256, B<=256, L<=64)");
  dt_options o;
  const dt_status ost = check_options(opts, &o);
  if (ost != DT_OK) return ost;
  dt_model *m = nullptr;
  dt_status st = dt_model_create(&m, emb, V, d_e, gru, head, weights_dtype);
  if (st != DT_OK) return st;
  st = dt_plan_create_from_model(plan, m, L, M, B, logits_dtype, max_batch, opts);
  model_release(m);  // the plan holds the only reference now (or none: freed)
  return st;
}

dt_status dt_plan_set_profiling(dt_plan *p, int enable) {
  if (!p) return fail(DT_ERR_NULL, "plan is required");
  if (enable && !p->ev) {
    p->ev = new (std::nothrow) hipEvent_t[4 * dt::kProfSlots]();
    if (!p->ev) return fail(DT_ERR_HIP, "host allocation failed");
    for (int i = 0; i < 4 * dt::kProfSlots; ++i) {
      hipError_t e = hipEventCreate(&p->ev[i]);
      if (e != hipSuccess) return hip_fail(e, "event create");
    }
  }
  if (enable && !p->stats) {
    const hipError_t e = hipMalloc(&p->stats, sizeof(int32_t) * 2 * p->max_batch);
    if (e != hipSuccess) return hip_fail(e, "stats buffer");
  }
  p->profiling = enable > 0 ? enable : 0;
  p->stats_batch = 0;
  p->profiled_calls = 0;
  p->calls_since = 0;
  return DT_OK;
}

dt_status dt_plan_stage_ms(dt_plan *p, float *ms) {
  if (!p || !ms) return fail(DT_ERR_NULL, "plan and ms are required");
  if (!p->ev || p->profiled_calls == 0)
    return fail(DT_ERR_SHAPE, "no profiled dt_build_tree call yet");
  const int n = p->profiled_calls < dt::kProfSlots ? p->profiled_calls : dt::kProfSlots;
  const int last = (p->profiled_calls - 1) % dt::kProfSlots;
  hipError_t e = hipEventSynchronize(p->ev[4 * last + 3]);
  double sum[2] = {0.0, 0.0};
  for (int c = 0; c < n && e == hipSuccess; ++c)
    for (int i = 0; i < 2 && e == hipSuccess; ++i) {
      float t = 0.0f;
      e = hipEventElapsedTime(&t, p->ev[4 * c + 2 * i], p->ev[4 * c + 2 * i + 1]);
      sum[i] += t;
    }
  if (e != hipSuccess) return hip_fail(e, "event timing");
  for (int i = 0; i < 2; ++i) ms[i] = (float)(sum[i] / n);
  return DT_OK;
}

dt_status dt_plan_set_adaptive_budget(dt_plan *p, float c_draft, const float *c_verify, int n) {
  if (!p) return fail(DT_ERR_NULL, "plan is required");
  if (!c_verify) {
    p->cost = nullptr;  // (the buffer stays allocated until the plan is destroyed)
    return DT_OK;
  }
  if (n != p->B + 1) return fail(DT_ERR_SHAPE, "c_verify needs B + 1 = %d entries, got %d", p->B + 1, n);
  if (p->frontier_w > 0)
    return fail(DT_ERR_UNSUPPORTED, "the adaptive budget applies to the heap builder (frontier_width 0)");
  float host[dt::kMaxB + 2];
  host[0] = c_draft;
  for (int i = 0; i < n; ++i) {
    const float den = c_draft + c_verify[i];
    if (!(den > 0.0f) || !(den < __builtin_huge_valf()))
      return fail(DT_ERR_SHAPE, "C_d + C_v(%d) = %g must be positive and finite", i, (double)den);
    host[1 + i] = c_verify[i];
  }
  if (!p->cost_buf) {
    const hipError_t e = hipMalloc(&p->cost_buf, sizeof(float) * (dt::kMaxB + 2));
    if (e != hipSuccess) return hip_fail(e, "cost buffer");
  }
  const hipError_t e = hipMemcpy(p->cost_buf, host, sizeof(float) * (n + 1), hipMemcpyHostToDevice);
  if (e != hipSuccess) return hip_fail(e, "cost copy");
  p->cost = p->cost_buf;
  return DT_OK;
}

dt_status dt_plan_expand_stats(dt_plan *p, int32_t *steps, int32_t *expanded, int n) {
  if (!p || !steps || !expanded) return fail(DT_ERR_NULL, "plan, steps and expanded are required");
  if (!p->stats || p->stats_batch == 0) return fail(DT_ERR_SHAPE, "no profiled dt_build_tree call yet");
  if (n < 1 || n > p->stats_batch)
    return fail(DT_ERR_SHAPE, "n %d outside [1, %d] (trees of the last profiled call)", n,
                p->stats_batch);
  hipError_t e0 = hipDeviceSynchronize();  // the profiled call may sit on any stream
  if (e0 != hipSuccess) return hip_fail(e0, "device synchronize");
  int32_t buf[2 * 256];
  for (int t0 = 0; t0 < n; t0 += 256) {
    const int m = n - t0 < 256 ? n - t0 : 256;
    const hipError_t e =
        hipMemcpy(buf, p->stats + 2 * t0, sizeof(int32_t) * 2 * m, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "stats copy");
    for (int i = 0; i < m; ++i) {
      steps[t0 + i] = buf[2 * i];
      expanded[t0 + i] = buf[2 * i + 1];
    }
  }
  return DT_OK;
}

void dt_plan_destroy(dt_plan *p) {
  if (!p) return;
  if (p->stats) (void)hipFree(p->stats);
  if (p->cost_buf) (void)hipFree(p->cost_buf);
  if (p->ev) {
    for (int i = 0; i < 4 * dt::kProfSlots; ++i)
      if (p->ev[i]) (void)hipEventDestroy(p->ev[i]);
    delete[] p->ev;
  }
  model_release(p->model);
  delete p;
}

dt_status dt_workspace_size(const dt_plan *plan, int batch, size_t *bytes) {
  if (!plan || !bytes) return fail(DT_ERR_NULL, "plan and bytes are required");
  if (batch < 1 || batch > plan->max_batch)
    return fail(DT_ERR_SHAPE, "batch %d outside [1, max_batch=%d]", batch, plan->max_batch);
  *bytes = dt::carve(plan, batch, nullptr).bytes;
  return DT_OK;
}

static dt_status check_build_args(const dt_plan *plan, const void *logits, int batch,
                                  const float *h0, float T, const dt_tree *out) {
  if (!plan || !logits || !out) return fail(DT_ERR_NULL, "plan, logits and out are required");
  if (!out->tokens || !out->parents || !out->depth || !out->position_ids || !out->mask ||
      !out->scores || !out->n_nodes || !out->status)
    return fail(DT_ERR_NULL, "every dt_tree output pointer is required");
  if (batch < 1 || batch > plan->max_batch)
    return fail(DT_ERR_SHAPE, "batch %d outside [1, max_batch=%d]", batch, plan->max_batch);
  if (!(T == T)) return fail(DT_ERR_SHAPE, "temperature is NaN");
  if (!aligned(logits, dsize(plan->ldt)) || (h0 && !aligned(h0, 4)) || !aligned(out->tokens, 4) ||
      !aligned(out->parents, 4) || !aligned(out->depth, 4) || !aligned(out->position_ids, 4) ||
      !aligned(out->scores, 4) || !aligned(out->n_nodes, 4) || !aligned(out->status, 4))
    return fail(DT_ERR_ALIGN, "logits and outputs must be naturally aligned");
  return DT_OK;
}

// The launches of one dt_build_tree call on a checked, large enough workspace.
static dt_status build_tree_on(dt_plan *plan, const void *logits, int batch, const float *h0,
                               float T, void *workspace, dt_tree *out, void *stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  const float inv_tau = T > 0.0f ? 1.0f / T : 1.0f;
  dt::Workspace ws = dt::carve(plan, batch, static_cast<char *>(workspace));
  const dt::ScanGeom g = dt::scan_geom(batch * plan->L, plan->V, plan->M);
  // profiling every n-th call: the events' own cost (a few us each) stays small.
  // Calls captured into a graph are neither profiled nor counted.
  bool prof = false;
  if (plan->profiling > 0) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    const hipError_t ce = hipStreamIsCapturing(s, &cs);
    if (ce != hipSuccess) return hip_fail(ce, "stream capture query");
    if (cs == hipStreamCaptureStatusNone) prof = (plan->calls_since++ % plan->profiling) == 0;
  }
  // profiled calls time each kernel from its start to its end
  hipEvent_t *ev = prof ? plan->ev + 4 * (plan->profiled_calls % dt::kProfSlots) : nullptr;
  // the scan kernel also clears the expansion launches' barrier counters
  const int nbar = (batch + dt::kSlotRows) * dt::kBarStride;
  hipError_t e = dt::launch_scan_chunks(logits, plan->ldt, g, inv_tau, ws, ws.bar, 2 * nbar, s,
                                        prof ? ev[0] : nullptr, prof ? ev[1] : nullptr);
  if (e != hipSuccess) return hip_fail(e, "scan launch");
  dt::ExpMode mode;
  if (plan->scorer == DT_SCORER_MARG) {
    mode.nocorr = 1;
  } else if (plan->scorer == DT_SCORER_STATIC) {
    // the greedy chain (k = 1, L pops) writes every depth's corrected menu;
    // the tree is then built from those menus
    dt::ExpMode chain;
    chain.menu_out = ws.menus;
    chain.emit = 0;
    chain.k = 1;
    chain.B = plan->L;
    e = dt::launch_expand(plan, batch, h0, inv_tau, ws, out, s, nullptr, nullptr, chain);
    if (e != hipSuccess) return hip_fail(e, "expand launch (greedy chain)");
    mode.nocorr = 1;
    mode.menu_in = ws.menus;
    mode.skip_merge = 1;
    mode.bar = ws.bar + nbar;
  }
  if (prof) {
    mode.stats = plan->stats;
    plan->stats_batch = batch;
  }
  e = dt::launch_expand(plan, batch, h0, inv_tau, ws, out, s, prof ? ev[2] : nullptr,
                        prof ? ev[3] : nullptr, mode);
  if (e != hipSuccess) return hip_fail(e, "expand launch");
  if (prof) plan->profiled_calls++;
  return DT_OK;
}

dt_status dt_build_tree(dt_plan *plan, const void *logits, int batch, const float *h0, float T,
                        void *workspace, size_t ws_bytes, dt_tree *out, void *stream) {
  const dt_status st = check_build_args(plan, logits, batch, h0, T, out);
  if (st != DT_OK) return st;
  const size_t need = dt::carve(plan, batch, nullptr).bytes;
  if (!workspace || ws_bytes < need)
    return fail(DT_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, workspace ? ws_bytes : 0);
  if (!aligned(workspace, 256)) return fail(DT_ERR_ALIGN, "workspace must be 256-byte aligned");
  return build_tree_on(plan, logits, batch, h0, T, workspace, out, stream);
}

dt_status dt_build_tree_noalloc(dt_plan *plan, const void *logits, int batch, const float *h0,
                                float T, dt_tree *out, void *stream) {
  const dt_status st = check_build_args(plan, logits, batch, h0, T, out);
  if (st != DT_OK) return st;
  const size_t need = dt::carve(plan, batch, nullptr).bytes;
  if (need > kScratchBytes)
    return fail(DT_ERR_WORKSPACE,
                "batch %d needs %zu bytes of workspace, more than the %zu-byte scratch of "
                "dt_build_tree_noalloc; use dt_build_tree with a workspace", batch, need,
                kScratchBytes);
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "device query");
  if (dev != plan->device)
    return fail(DT_ERR_SHAPE, "the current device (%d) is not the plan's device (%d)", dev,
                plan->device);
  void *ws = nullptr;
  e = scratch_address(dev, &ws);  // resolved when the plan was created: a table lookup
  if (e != hipSuccess) return hip_fail(e, "scratch address");
  return build_tree_on(plan, logits, batch, h0, T, ws, out, stream);
}

dt_status dt_scan_workspace_size(int rows, int V, int M, size_t *bytes) {
  if (!bytes) return fail(DT_ERR_NULL, "bytes is required");
  if (rows < 1 || V < 1 || M < 1 || M > V) return fail(DT_ERR_SHAPE, "need rows, V >= 1 and 1 <= M <= V");
  if (M > dt::kMaxM) return fail(DT_ERR_UNSUPPORTED, "M must be <= 256");
  if (dt::merge_lds_bytes(dt::scan_geom(rows, V, M)) > (size_t)dt::kMergeLdsMax)
    return fail(DT_ERR_UNSUPPORTED, "V and M too large for the row merge");
  *bytes = dt::scan_bytes(dt::scan_geom(rows, V, M));
  return DT_OK;
}

dt_status dt_scan_topm(const void *logits, int rows, int V, int logits_dtype, int M, float T,
                       int32_t *ids, float *vals, float *tail_lse, int32_t *row_flags,
                       void *workspace, size_t ws_bytes, void *stream) {
  if (!logits || !ids || !vals || !tail_lse || !row_flags)
    return fail(DT_ERR_NULL, "logits and every output are required");
  if (!valid_dtype(logits_dtype)) return fail(DT_ERR_DTYPE, "dtype must be DT_F32 or DT_BF16");
  if (rows < 1 || V < 1 || M < 1 || M > V) return fail(DT_ERR_SHAPE, "need rows, V >= 1 and 1 <= M <= V");
  if (M > dt::kMaxM) return fail(DT_ERR_UNSUPPORTED, "M must be <= 256");
  if (!(T == T)) return fail(DT_ERR_SHAPE, "temperature is NaN");
  const dt::ScanGeom g = dt::scan_geom(rows, V, M);
  if (dt::merge_lds_bytes(g) > (size_t)dt::kMergeLdsMax)
    return fail(DT_ERR_UNSUPPORTED, "V and M too large for the row merge");
  const size_t need = dt::scan_bytes(g);
  if (!workspace || ws_bytes < need)
    return fail(DT_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, workspace ? ws_bytes : 0);
  if (!aligned(workspace, 256)) return fail(DT_ERR_ALIGN, "workspace must be 256-byte aligned");
  if (!aligned(logits, dsize(logits_dtype)) || !aligned(ids, 4) || !aligned(vals, 4) ||
      !aligned(tail_lse, 4) || !aligned(row_flags, 4))
    return fail(DT_ERR_ALIGN, "logits and outputs must be naturally aligned");
  dt::Workspace ws{};
  dt::carve_scan(static_cast<char *>(workspace), g, &ws);
  ws.cand = ids;
  ws.candv = vals;
  ws.tail = tail_lse;
  ws.row_flag = row_flags;
  const float inv_tau = T > 0.0f ? 1.0f / T : 1.0f;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = dt::launch_scan_chunks(logits, logits_dtype, g, inv_tau, ws, nullptr, 0, s);
  if (e == hipSuccess) e = dt::launch_scan_merge(g, inv_tau, ws, s);
  if (e != hipSuccess) return hip_fail(e, "scan launch");
  return DT_OK;
}

// Domino's head on the expansion kernel (the default path's member split and
// speculative expansion): G members per tree, member j owning ranks
// [j rank / G, (j + 1) rank / G).  Returns G, or 0 when the shape is outside
// that kernel's envelope and the one-workgroup head kernel builds the tree.
static int head_fast_group(const dt_plan *p, int batch, const dt_domino_head *hd, int maxlds) {
  const int G = dt::expand_group_size(p, batch);
  if (hd->rank % (16 * G) != 0) return 0;
  const int rj = hd->rank / G;
  if (rj != 16 && rj != 32 && rj != 64) return 0;  // whole MFMA tiles; 64 % (lanes per W_2 row) == 0
  const int es = dsize(p->wdt);
  if ((size_t)p->V * hd->rank * es >= ((size_t)1 << 31)) return 0;  // buffer offsets of W_2 rows
  const dt::ScanGeom g = dt::scan_geom(batch * p->L, p->V, p->M);
  if (dt::expand_lds_bytes(p->d_h, G, p->M, g.nchunks, p->L, rj, es) > (size_t)maxlds) return 0;
  return G;
}

struct HeadFastWs {
  dt::Workspace ws;  // the default path's (scan lists, states, exchange, counters)
  float *a;          // [batch * L][rank] W_1^H H
  float *hpart;      // [batch][2][G][16][rank] partial W_1^S S of each member
  size_t bytes;
};
static HeadFastWs carve_head_fast(const dt_plan *p, int batch, int rank, int G, char *base) {
  HeadFastWs h;
  h.ws = dt::carve(p, batch, base);
  size_t o = h.ws.bytes;
  h.a = base ? reinterpret_cast<float *>(base + o) : nullptr;
  o += dt::align_up((size_t)batch * p->L * rank * sizeof(float), 256);
  h.hpart = base ? reinterpret_cast<float *>(base + o) : nullptr;
  o += dt::align_up((size_t)batch * 2 * G * 16 * rank * sizeof(float), 256);
  h.bytes = o;
  return h;
}

// checks shared by dt_head_workspace_size and dt_build_tree_head; *G the
// fast path's group size (0: the one-workgroup head kernel)
static dt_status head_check(const dt_plan *plan, int batch, const dt_domino_head *hd, int *G) {
  if (!plan || !hd) return fail(DT_ERR_NULL, "plan and head are required");
  if (!hd->w1 || !hd->w2) return fail(DT_ERR_NULL, "head.w1 and head.w2 are required");
  if (batch < 1 || batch > plan->max_batch)
    return fail(DT_ERR_SHAPE, "batch %d outside [1, max_batch=%d]", batch, plan->max_batch);
  if (hd->d_H < 8 || hd->d_H > 8192 || hd->d_H % 8 != 0 || hd->rank < 8 || hd->rank > 1024 ||
      hd->rank % 8 != 0)
    return fail(DT_ERR_SHAPE, "need 8 <= d_H <= 8192 and 8 <= rank <= 1024, multiples of 8 (d_H=%d rank=%d)",
                hd->d_H, hd->rank);
  if (plan->scorer != DT_SCORER_COND || plan->frontier_w != 0)
    return fail(DT_ERR_UNSUPPORTED,
                "the Domino head needs a plan created with DT_SCORER_COND and frontier_width 0");
  int dev = 0, maxlds = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&maxlds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return hip_fail(e, "device query");
  *G = head_fast_group(plan, batch, hd, maxlds);
  if (*G > 0) return DT_OK;
  // the one-workgroup head kernel
  const dt::ScanGeom g = dt::scan_geom(batch * plan->L, plan->V, plan->M);
  if (!dt::sel::wave_merge_fits(g.nchunks, plan->M))
    return fail(DT_ERR_UNSUPPORTED, "the Domino head needs M <= 64 and <= 16 scan segments per row (M=%d, %d)",
                plan->M, g.nchunks);
  if ((size_t)plan->k * (plan->B + 1) > (size_t)dt::kHeadCap)
    return fail(DT_ERR_UNSUPPORTED, "k * (B + 1) = %d exceeds the heap's %d entries",
                plan->k * (plan->B + 1), dt::kHeadCap);
  const size_t lds = dt::head_lds_bytes(plan->L, plan->B, plan->d_h, hd->rank);
  if (lds > (size_t)maxlds)
    return fail(DT_ERR_UNSUPPORTED, "the Domino head needs %zu bytes of LDS, the device has %d", lds, maxlds);
  return DT_OK;
}

static size_t head_ws_bytes(const dt_plan *plan, int batch, const dt_domino_head *hd, int G) {
  return G > 0 ? carve_head_fast(plan, batch, hd->rank, G, nullptr).bytes
               : dt::carve_head(plan, batch, hd->rank, nullptr).bytes;
}

dt_status dt_head_workspace_size(const dt_plan *plan, int batch, const dt_domino_head *head,
                                 size_t *bytes) {
  if (!bytes) return fail(DT_ERR_NULL, "bytes is required");
  int G = 0;
  const dt_status st = head_check(plan, batch, head, &G);
  if (st != DT_OK) return st;
  *bytes = head_ws_bytes(plan, batch, head, G);
  return DT_OK;
}

dt_status dt_build_tree_head(dt_plan *plan, const void *logits, int batch, const void *H,
                             const dt_domino_head *head, const float *h0, float T, void *workspace,
                             size_t ws_bytes, dt_tree *out, void *stream) {
  if (!plan || !logits || !H || !out) return fail(DT_ERR_NULL, "plan, logits, H and out are required");
  if (!out->tokens || !out->parents || !out->depth || !out->position_ids || !out->mask ||
      !out->scores || !out->n_nodes || !out->status)
    return fail(DT_ERR_NULL, "every dt_tree output pointer is required");
  int G = 0;
  const dt_status st = head_check(plan, batch, head, &G);
  if (st != DT_OK) return st;
  if (!(T == T)) return fail(DT_ERR_SHAPE, "temperature is NaN");
  const size_t need = head_ws_bytes(plan, batch, head, G);
  if (!workspace || ws_bytes < need)
    return fail(DT_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, workspace ? ws_bytes : 0);
  if (!aligned(workspace, 256)) return fail(DT_ERR_ALIGN, "workspace must be 256-byte aligned");
  if (!aligned(head->w1, 16) || !aligned(head->w2, 16) || !aligned(H, 16))
    return fail(DT_ERR_ALIGN, "head.w1, head.w2 and H must be 16-byte aligned");
  if (!aligned(logits, dsize(plan->ldt)) || (h0 && !aligned(h0, 4)) || !aligned(out->tokens, 4) ||
      !aligned(out->parents, 4) || !aligned(out->depth, 4) || !aligned(out->position_ids, 4) ||
      !aligned(out->scores, 4) || !aligned(out->n_nodes, 4) || !aligned(out->status, 4))
    return fail(DT_ERR_ALIGN, "logits and outputs must be naturally aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const float inv_tau = T > 0.0f ? 1.0f / T : 1.0f;
  const dt::ScanGeom g = dt::scan_geom(batch * plan->L, plan->V, plan->M);
  // stage timing as in dt_build_tree: stage 0 the scan, stage 1 the tree kernel
  bool prof = false;
  if (plan->profiling > 0) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    const hipError_t ce = hipStreamIsCapturing(s, &cs);
    if (ce != hipSuccess) return hip_fail(ce, "stream capture query");
    if (cs == hipStreamCaptureStatusNone) prof = (plan->calls_since++ % plan->profiling) == 0;
  }
  hipEvent_t *ev = prof ? plan->ev + 4 * (plan->profiled_calls % dt::kProfSlots) : nullptr;
  if (G > 0) {
    // the scan (clearing the expansion's barrier counters; its extra
    // workgroups compute a_d = W_1^H H_d), then the default path's expansion
    // kernel with Domino's head
    const HeadFastWs hf = carve_head_fast(plan, batch, head->rank, G, static_cast<char *>(workspace));
    const int nbar = (batch + dt::kSlotRows) * dt::kBarStride;
    const dt::HeadProj hp = dt::head_proj_args(plan, batch * plan->L, H, *head, hf.a);
    hipError_t e = dt::launch_scan_chunks(logits, plan->ldt, g, inv_tau, hf.ws, hf.ws.bar, 2 * nbar, s,
                                          prof ? ev[0] : nullptr, prof ? ev[1] : nullptr, &hp);
    if (e != hipSuccess) return hip_fail(e, "scan launch");
    dt::HeadIn hin{head->w1, head->w2, hf.a, hf.hpart, head->rank, head->d_H};
    dt::ExpMode mode;
    mode.head = &hin;
    if (prof) {
      mode.stats = plan->stats;
      plan->stats_batch = batch;
    }
    e = dt::launch_expand(plan, batch, h0, inv_tau, hf.ws, out, s, prof ? ev[2] : nullptr,
                          prof ? ev[3] : nullptr, mode);
    if (e != hipSuccess) return hip_fail(e, "expand launch (Domino head)");
    if (prof) plan->profiled_calls++;
    return DT_OK;
  }
  const dt::HeadWorkspace hw = dt::carve_head(plan, batch, head->rank, static_cast<char *>(workspace));
  const dt::HeadProj hp = dt::head_proj_args(plan, batch * plan->L, H, *head, hw.a);
  hipError_t e = dt::launch_scan_chunks(logits, plan->ldt, g, inv_tau, hw.scan, nullptr, 0, s,
                                        prof ? ev[0] : nullptr, prof ? ev[1] : nullptr, &hp);
  if (e != hipSuccess) return hip_fail(e, "scan launch");
  e = dt::launch_head(plan, batch, H, *head, h0, inv_tau, hw, out, s, prof ? ev[2] : nullptr,
                      prof ? ev[3] : nullptr);
  if (e != hipSuccess) return hip_fail(e, "head launch");
  if (prof) plan->profiled_calls++;
  return DT_OK;
}

}  // extern "C"
