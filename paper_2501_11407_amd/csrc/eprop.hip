// Host side of the e-prop library: C ABI (include/eprop.h), workspace
// layout and the per-step launch schedule.  No device memory is allocated
// here: every buffer is carved from the caller's workspace.
#include "../../include/eprop.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "kernels.h"

namespace {

thread_local std::string g_last_error = "";

size_t round_up(size_t v, size_t m) { return (v + m - 1) / m * m; }

// Split-K choice for a GEMM of M x N over K (multiple of 16): enough waves
// to cover the chip (~1024), at most max_splits, chunks a multiple of 16.
void choose_splits(int M, int N, int K, int max_splits, int* splits, int* k_chunk) {
  const long long tiles = (long long)((M + 31) / 32) * ((N + 31) / 32);
  long long want = std::max<long long>(1, (1024 + tiles - 1) / tiles);
  want = std::min<long long>(want, std::max(1, K / 16));
  want = std::min<long long>(want, max_splits);
  int kc = (int)round_up((K + want - 1) / want, 16);
  kc = std::max(kc, 16);
  *k_chunk = kc;
  *splits = (K + kc - 1) / kc;
}

struct Layer {
  int n_inl = 0, n_pre = 0;
  // padded extents
  int kpad = 0;   // n_pre rounded to 16: drive GEMM K and row stride of P, Wp
  int bpad = 0;   // batch rounded to 32: rows of P and Zf
  int npad = 0;   // n_rec rounded to 32: rows of Wp
  int nrk = 0;    // n_rec rounded to 16: readout GEMM K, row stride of Zf, Wop
  int kout = 0;   // n_out rounded to 32: rows of Wop
  int ldj = 0;    // n_rec rounded to 4: row stride of per-neuron buffers and traces
  int lda = 0;    // n_adaptive rounded to 4: row stride of epsa
  int ldz = 0;    // batch rounded to 4: row stride of zbarT
  int s_drive = 1, kc_drive = 16, s_out = 1, kc_out = 16;
  const float* W_src = nullptr;
  const float* Wout_src = nullptr;
  float *Wp, *Wop, *P, *zbarT, *Ipart, *v, *a, *Zf, *psi, *L, *ztil, *Ypart, *y, *delta;
  uint8_t* z[2];
  double *lossacc, *acc, *accout;
  float *ebar, *epsa;
};

struct Plan {
  eprop_config cfg;
  std::vector<Layer> layers;
  int* err_flag = nullptr;
  size_t bytes = 0;
};

bool valid_config(const eprop_config* c, std::string* why) {
  if (!c) { *why = "config is NULL"; return false; }
  if (c->n_layers != 1 && c->n_layers != 2) { *why = "n_layers must be 1 or 2"; return false; }
  if (c->batch < 1 || c->n_in < 1 || c->n_rec < 1 || c->n_out < 1) {
    *why = "batch, n_in, n_rec and n_out must be >= 1";
    return false;
  }
  if (c->batch > 65535) { *why = "batch must be <= 65535"; return false; }
  if (c->n_out > 8192) { *why = "n_out must be <= 8192"; return false; }
  if (c->recurrent != 0 && c->recurrent != 1) { *why = "recurrent must be 0 or 1"; return false; }
  if (c->n_adaptive < 0 || c->n_adaptive > c->n_rec) {
    *why = "n_adaptive must be in [0, n_rec]";
    return false;
  }
  const float k[] = {c->alpha, c->rho, c->kappa, c->thr, c->beta, c->gamma};
  for (float v : k)
    if (!std::isfinite(v)) { *why = "constants must be finite"; return false; }
  if (!(c->thr > 0.0f)) { *why = "thr must be > 0"; return false; }
  const long long n_pre_max = (long long)std::max(c->n_in, c->n_rec) + (c->recurrent ? c->n_rec : 0);
  if (n_pre_max > (1LL << 30) / 4) { *why = "presynaptic dimension too large"; return false; }
  return true;
}

// Lays the workspace out (base == nullptr: sizing only).
void make_plan(const eprop_config& c, char* base, Plan* plan) {
  plan->cfg = c;
  plan->layers.assign(c.n_layers, Layer());
  size_t off = 0;
  auto take = [&](size_t bytes) -> char* {
    off = round_up(off, 256);
    char* p = base ? base + off : nullptr;
    off += round_up(std::max<size_t>(bytes, 1), 256);
    return p;
  };
  const size_t B = c.batch, N = c.n_rec, K = c.n_out;
  plan->err_flag = (int*)take(sizeof(int));
  for (int l = 0; l < c.n_layers; ++l) {
    Layer& L = plan->layers[l];
    L.n_inl = (l == 0) ? c.n_in : c.n_rec;
    L.n_pre = L.n_inl + (c.recurrent ? c.n_rec : 0);
    L.kpad = (int)round_up(L.n_pre, 16);
    L.bpad = (int)round_up(B, 32);
    L.npad = (int)round_up(N, 32);
    L.nrk = (int)round_up(N, 16);
    L.kout = (int)round_up(K, 32);
    L.ldj = (int)round_up(N, 4);
    L.lda = (int)round_up(std::max(c.n_adaptive, 1), 4);
    L.ldz = (int)round_up(B, 4);
    choose_splits(c.batch, c.n_rec, L.kpad, 16, &L.s_drive, &L.kc_drive);
    choose_splits(c.batch, c.n_out, L.nrk, 16, &L.s_out, &L.kc_out);
    const size_t np = L.n_pre;
    L.Wp = (float*)take(sizeof(float) * L.npad * L.kpad);
    L.Wop = (float*)take(sizeof(float) * L.kout * L.nrk);
    L.P = (float*)take(sizeof(float) * L.bpad * L.kpad);
    L.zbarT = (float*)take(sizeof(float) * np * L.ldz);
    L.Ipart = (float*)take(sizeof(float) * L.s_drive * B * L.ldj);
    L.v = (float*)take(sizeof(float) * B * N);
    L.a = (float*)take(sizeof(float) * B * N);
    L.z[0] = (uint8_t*)take(B * N);
    L.z[1] = (uint8_t*)take(B * N);
    L.Zf = (float*)take(sizeof(float) * L.bpad * L.nrk);
    L.psi = (float*)take(sizeof(float) * B * L.ldj);
    L.L = (float*)take(sizeof(float) * B * L.ldj);
    L.ztil = (float*)take(sizeof(float) * B * L.ldj);
    L.Ypart = (float*)take(sizeof(float) * L.s_out * B * K);
    L.y = (float*)take(sizeof(float) * B * K);
    L.delta = (float*)take(sizeof(float) * B * K);
    L.lossacc = (double*)take(sizeof(double) * B);
    L.acc = (double*)take(sizeof(double) * np * L.ldj);
    L.accout = (double*)take(sizeof(double) * K * L.ldj);
    L.ebar = (float*)take(sizeof(float) * B * np * L.ldj);
    L.epsa = (float*)take(c.n_adaptive > 0 ? sizeof(float) * B * np * L.lda : 0);
  }
  plan->bytes = round_up(off, 256);
}

}  // namespace

struct eprop_ctx {
  Plan plan;
  char* ws = nullptr;
  size_t ws_bytes = 0;
  hipStream_t stream = nullptr;
  long long t = 0;      // steps since the last reset
  int cur = 0;          // index of z^{t-1} in Layer::z
  bool alive = false;
  std::string err;
  // profiling of the eligibility kernel
  bool prof = false;
  std::vector<hipEvent_t> ev;
  int prof_max = 0, prof_n = 0;
};

namespace {

int fail(eprop_ctx* ctx, int code, const std::string& msg) {
  if (ctx) ctx->err = msg; else g_last_error = msg;
  return code;
}

int check(eprop_ctx* ctx, hipError_t e, const char* what) {
  if (e == hipSuccess) return EPROP_OK;
  return fail(ctx, EPROP_EDEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

int pack_weights(eprop_ctx* ctx) {
  for (Layer& L : ctx->plan.layers) {
    const eprop_config& c = ctx->plan.cfg;
    int rc = check(ctx, eprop::launch_pack(L.W_src, c.n_rec, L.n_pre, L.Wp, L.kpad, L.npad, ctx->stream),
                   "weight packing");
    if (rc) return rc;
    rc = check(ctx, eprop::launch_pack(L.Wout_src, c.n_out, c.n_rec, L.Wop, L.nrk, L.kout, ctx->stream),
               "readout weight packing");
    if (rc) return rc;
  }
  return EPROP_OK;
}

// Zeroes the small state.  Traces and accumulators are not cleared: the
// first step after a reset treats them as zero without reading them.
int clear_state(eprop_ctx* ctx) {
  const eprop_config& c = ctx->plan.cfg;
  const size_t B = c.batch, N = c.n_rec, K = c.n_out;
  hipStream_t s = ctx->stream;
  int rc = check(ctx, hipMemsetAsync(ctx->plan.err_flag, 0, sizeof(int), s), "reset");
  for (Layer& L : ctx->plan.layers) {
    if (rc) return rc;
    hipError_t e = hipSuccess;
    e = e ? e : hipMemsetAsync(L.zbarT, 0, sizeof(float) * L.n_pre * L.ldz, s);
    e = e ? e : hipMemsetAsync(L.v, 0, sizeof(float) * B * N, s);
    e = e ? e : hipMemsetAsync(L.a, 0, sizeof(float) * B * N, s);
    e = e ? e : hipMemsetAsync(L.z[0], 0, B * N, s);
    e = e ? e : hipMemsetAsync(L.z[1], 0, B * N, s);
    e = e ? e : hipMemsetAsync(L.ztil, 0, sizeof(float) * B * L.ldj, s);
    e = e ? e : hipMemsetAsync(L.y, 0, sizeof(float) * B * K, s);
    e = e ? e : hipMemsetAsync(L.lossacc, 0, sizeof(double) * B, s);
    rc = check(ctx, e, "reset");
  }
  ctx->t = 0;
  ctx->cur = 0;
  return rc;
}

int do_step(eprop_ctx* ctx, const uint8_t* x_t, const int32_t* labels, uint32_t* spikes_t) {
  const eprop_config& c = ctx->plan.cfg;
  hipStream_t s = ctx->stream;
  const int prev = ctx->cur, now = ctx->cur ^ 1;
  const int W32 = (c.n_rec + 31) / 32;
  const int first = ctx->t == 0;
  int rc;
  for (int l = 0; l < c.n_layers; ++l) {
    Layer& L = ctx->plan.layers[l];
    eprop::PresynArgs pa;
    pa.in = (l == 0) ? x_t : ctx->plan.layers[l - 1].z[now];
    pa.zprev = L.z[prev];
    pa.P = L.P; pa.zbarT = L.zbarT;
    pa.B = c.batch; pa.n_inl = L.n_inl; pa.n_rec = c.n_rec; pa.n_pre = L.n_pre;
    pa.ldp = L.kpad; pa.ldz = L.ldz; pa.alpha = c.alpha;
    if ((rc = check(ctx, eprop::launch_presyn(pa, s), "presynaptic kernel"))) return rc;

    eprop::GemmArgs g;
    g.A = L.P; g.Bm = L.Wp; g.C = L.Ipart;
    g.M = c.batch; g.N = c.n_rec; g.K = L.kpad; g.lda = L.kpad; g.ldb = L.kpad; g.ldc = L.ldj;
    g.splits = L.s_drive; g.k_chunk = L.kc_drive; g.split_stride = (size_t)c.batch * L.ldj;
    if ((rc = check(ctx, eprop::launch_gemm_nt(g, s), "drive GEMM"))) return rc;

    eprop::NeuronArgs na;
    na.Ipart = L.Ipart; na.splits = L.s_drive; na.split_stride = g.split_stride; na.ldI = L.ldj;
    na.v = L.v; na.a = L.a; na.zprev = L.z[prev]; na.zcur = L.z[now];
    na.Zf = L.Zf; na.ldzf = L.nrk; na.psi = L.psi; na.ldj = L.ldj;
    na.spikes = spikes_t ? spikes_t + (size_t)l * c.batch * W32 : nullptr;
    na.W32 = W32; na.B = c.batch; na.n_rec = c.n_rec; na.n_adaptive = c.n_adaptive;
    na.alpha = c.alpha; na.rho = c.rho; na.thr = c.thr; na.beta = c.beta;
    na.gamma_over_thr = c.gamma / c.thr;
    if ((rc = check(ctx, eprop::launch_neuron(na, s), "neuron kernel"))) return rc;
  }
  for (int l = 0; l < c.n_layers; ++l) {
    Layer& L = ctx->plan.layers[l];
    eprop::GemmArgs g;
    g.A = L.Zf; g.Bm = L.Wop; g.C = L.Ypart;
    g.M = c.batch; g.N = c.n_out; g.K = L.nrk; g.lda = L.nrk; g.ldb = L.nrk; g.ldc = c.n_out;
    g.splits = L.s_out; g.k_chunk = L.kc_out; g.split_stride = (size_t)c.batch * c.n_out;
    if ((rc = check(ctx, eprop::launch_gemm_nt(g, s), "readout GEMM"))) return rc;

    eprop::ReadoutArgs ra;
    ra.Ypart = L.Ypart; ra.splits = L.s_out; ra.split_stride = g.split_stride; ra.ldY = c.n_out;
    ra.y = L.y; ra.delta = L.delta; ra.labels = labels; ra.Wout = L.Wop; ra.ldo = L.nrk;
    ra.zcur = L.z[now]; ra.L = L.L; ra.ztil = L.ztil; ra.ldj = L.ldj; ra.lossacc = L.lossacc;
    ra.err_flag = ctx->plan.err_flag; ra.B = c.batch; ra.K = c.n_out; ra.n_rec = c.n_rec;
    ra.kappa = c.kappa;
    if ((rc = check(ctx, eprop::launch_readout(ra, s), "readout kernel"))) return rc;

    eprop::DwoutArgs da;
    da.delta = L.delta; da.ztil = L.ztil; da.ldj = L.ldj; da.accout = L.accout; da.ld_acc = L.ldj;
    da.B = c.batch; da.K = c.n_out; da.n_rec = c.n_rec; da.first = first;
    if ((rc = check(ctx, eprop::launch_dwout(da, s), "readout gradient kernel"))) return rc;

    eprop::TraceArgs ta;
    ta.ebar = L.ebar; ta.epsa = L.epsa; ta.acc = L.acc; ta.zbarT = L.zbarT; ta.ldz = L.ldz;
    ta.psi = L.psi; ta.L = L.L; ta.B = c.batch; ta.n_pre = L.n_pre; ta.n_post = c.n_rec;
    ta.ldj = L.ldj; ta.n_adaptive = c.n_adaptive; ta.lda = L.lda;
    ta.kappa = c.kappa; ta.rho = c.rho; ta.beta = c.beta; ta.first = first;
    const bool timed = ctx->prof && ctx->prof_n < ctx->prof_max;
    if (timed && (rc = check(ctx, hipEventRecord(ctx->ev[2 * ctx->prof_n], s), "event record")))
      return rc;
    if ((rc = check(ctx, eprop::launch_trace(ta, s), "eligibility kernel"))) return rc;
    if (timed) {
      if ((rc = check(ctx, hipEventRecord(ctx->ev[2 * ctx->prof_n + 1], s), "event record")))
        return rc;
      ctx->prof_n++;
    }
  }
  ctx->cur = now;
  ctx->t++;
  return EPROP_OK;
}

bool usable(const eprop_ctx* ctx) { return ctx && ctx->alive; }

}  // namespace

extern "C" {

size_t eprop_workspace_bytes(const eprop_config* cfg) {
  std::string why;
  if (!valid_config(cfg, &why)) {
    g_last_error = why;
    return 0;
  }
  Plan p;
  make_plan(*cfg, nullptr, &p);
  return p.bytes;
}

int eprop_init(const eprop_config* cfg, void* d_workspace, size_t ws_bytes,
               const float* const* d_weights, void* hip_stream, eprop_ctx** out) {
  if (!out) return fail(nullptr, EPROP_EINVAL, "out is NULL");
  *out = nullptr;
  std::string why;
  if (!valid_config(cfg, &why)) return fail(nullptr, EPROP_EINVAL, why);
  if (!d_workspace || !d_weights) return fail(nullptr, EPROP_EINVAL, "workspace or weights is NULL");
  if (((uintptr_t)d_workspace) % 256 != 0)
    return fail(nullptr, EPROP_EINVAL, "workspace must be 256-byte aligned");
  for (int k = 0; k < 2 * cfg->n_layers; ++k)
    if (!d_weights[k]) return fail(nullptr, EPROP_EINVAL, "a weight pointer is NULL");
  Plan probe;
  make_plan(*cfg, nullptr, &probe);
  if (ws_bytes < probe.bytes)
    return fail(nullptr, EPROP_ENOSPACE,
                "workspace too small: need " + std::to_string(probe.bytes) + " bytes");
  eprop_ctx* ctx = new eprop_ctx();
  ctx->ws = (char*)d_workspace;
  ctx->ws_bytes = ws_bytes;
  ctx->stream = (hipStream_t)hip_stream;
  make_plan(*cfg, ctx->ws, &ctx->plan);
  for (int l = 0; l < cfg->n_layers; ++l) {
    ctx->plan.layers[l].W_src = d_weights[2 * l];
    ctx->plan.layers[l].Wout_src = d_weights[2 * l + 1];
  }
  // Padding of every buffer must read as zero; clear the whole layout once.
  int rc = check(ctx, hipMemsetAsync(ctx->ws, 0, ctx->plan.bytes, ctx->stream), "workspace clear");
  if (!rc) rc = pack_weights(ctx);
  if (!rc) rc = clear_state(ctx);
  if (rc) {
    g_last_error = ctx->err;
    delete ctx;
    return rc;
  }
  ctx->alive = true;
  *out = ctx;
  return EPROP_OK;
}

int eprop_step(eprop_ctx* ctx, const uint8_t* d_x_t, const int32_t* d_labels, uint32_t* d_spikes_t) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (!d_x_t || !d_labels) return fail(ctx, EPROP_EINVAL, "x or labels is NULL");
  return do_step(ctx, d_x_t, d_labels, d_spikes_t);
}

int eprop_run_sequence(eprop_ctx* ctx, const uint8_t* d_x, int32_t T, const int32_t* d_labels,
                       uint32_t* d_spikes) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (!d_x || !d_labels) return fail(ctx, EPROP_EINVAL, "x or labels is NULL");
  if (T < 1) return fail(ctx, EPROP_EINVAL, "T must be >= 1");
  const eprop_config& c = ctx->plan.cfg;
  const size_t x_step = (size_t)c.batch * c.n_in;
  const size_t s_step = (size_t)c.n_layers * c.batch * ((c.n_rec + 31) / 32);
  for (int32_t t = 0; t < T; ++t) {
    int rc = do_step(ctx, d_x + t * x_step, d_labels, d_spikes ? d_spikes + t * s_step : nullptr);
    if (rc) return rc;
  }
  return EPROP_OK;
}

int eprop_get_grads(eprop_ctx* ctx, float* const* d_grads, double* d_loss) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (!d_grads) return fail(ctx, EPROP_EINVAL, "grads is NULL");
  const eprop_config& c = ctx->plan.cfg;
  for (int k = 0; k < 2 * c.n_layers; ++k)
    if (!d_grads[k]) return fail(ctx, EPROP_EINVAL, "a gradient pointer is NULL");
  for (int l = 0; l < c.n_layers; ++l) {
    Layer& L = ctx->plan.layers[l];
    eprop::GradsArgs g;
    g.acc = L.acc; g.ldj = L.ldj; g.dW = d_grads[2 * l]; g.n_pre = L.n_pre; g.n_post = c.n_rec;
    g.n_inl = L.n_inl; g.recurrent = c.recurrent;
    g.accout = L.accout; g.ld_acc = L.ldj; g.dWout = d_grads[2 * l + 1]; g.K = c.n_out;
    g.valid = ctx->t > 0;
    int rc = check(ctx, eprop::launch_grads(g, ctx->stream), "gradient read-out");
    if (rc) return rc;
  }
  if (d_loss) {
    const Layer& L0 = ctx->plan.layers[0];
    const size_t stride = c.n_layers > 1 ? (size_t)(ctx->plan.layers[1].lossacc - L0.lossacc) : 0;
    int rc = check(ctx, eprop::launch_loss(L0.lossacc, c.batch, c.n_layers, stride, d_loss, ctx->stream),
                   "loss read-out");
    if (rc) return rc;
  }
  return EPROP_OK;
}

int eprop_reset(eprop_ctx* ctx) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  int rc = pack_weights(ctx);
  if (!rc) rc = clear_state(ctx);
  return rc;
}

int eprop_status(eprop_ctx* ctx) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  int flag = 0;
  int rc = check(ctx, hipMemcpyAsync(&flag, ctx->plan.err_flag, sizeof(int), hipMemcpyDeviceToHost,
                                     ctx->stream), "status read");
  if (!rc) rc = check(ctx, hipStreamSynchronize(ctx->stream), "stream synchronize");
  if (rc) return rc;
  if (flag) return fail(ctx, EPROP_ESTATE, "a label was outside [0, n_out)");
  return EPROP_OK;
}

void eprop_destroy(eprop_ctx* ctx) {
  if (!ctx) return;
  for (hipEvent_t e : ctx->ev) (void)hipEventDestroy(e);
  ctx->alive = false;
  delete ctx;
}

const char* eprop_last_error(const eprop_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_last_error.c_str();
}

int eprop_profile_begin(eprop_ctx* ctx, int32_t max_launches) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (max_launches < 1) return fail(ctx, EPROP_EINVAL, "max_launches must be >= 1");
  while ((int)ctx->ev.size() < 2 * max_launches) {
    hipEvent_t e;
    int rc = check(ctx, hipEventCreate(&e), "event create");
    if (rc) return rc;
    ctx->ev.push_back(e);
  }
  ctx->prof = true;
  ctx->prof_max = max_launches;
  ctx->prof_n = 0;
  return EPROP_OK;
}

int eprop_profile_end(eprop_ctx* ctx, double* total_ms, int32_t* n_launches) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (!total_ms || !n_launches) return fail(ctx, EPROP_EINVAL, "output pointer is NULL");
  int rc = check(ctx, hipStreamSynchronize(ctx->stream), "stream synchronize");
  if (rc) return rc;
  double sum = 0.0;
  for (int k = 0; k < ctx->prof_n; ++k) {
    float ms = 0.0f;
    rc = check(ctx, hipEventElapsedTime(&ms, ctx->ev[2 * k], ctx->ev[2 * k + 1]), "event time");
    if (rc) return rc;
    sum += ms;
  }
  *total_ms = sum;
  *n_launches = ctx->prof_n;
  ctx->prof = false;
  ctx->prof_n = 0;
  return EPROP_OK;
}

int eprop_debug_buffer(eprop_ctx* ctx, int32_t layer, int32_t which, const float** d_ptr,
                       int64_t* cols, int64_t* ld) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (!d_ptr || !cols || !ld) return fail(ctx, EPROP_EINVAL, "output pointer is NULL");
  const eprop_config& c = ctx->plan.cfg;
  if (layer < 0 || layer >= c.n_layers) return fail(ctx, EPROP_EINVAL, "bad layer");
  const Layer& L = ctx->plan.layers[layer];
  switch (which) {
    case 0: *d_ptr = L.v; *cols = c.n_rec; *ld = c.n_rec; break;
    case 1: *d_ptr = L.a; *cols = c.n_rec; *ld = c.n_rec; break;
    case 2: *d_ptr = L.psi; *cols = c.n_rec; *ld = L.ldj; break;
    case 3: *d_ptr = L.L; *cols = c.n_rec; *ld = L.ldj; break;
    case 4: *d_ptr = L.y; *cols = c.n_out; *ld = c.n_out; break;
    default: return fail(ctx, EPROP_EINVAL, "unknown buffer");
  }
  return EPROP_OK;
}

}  // extern "C"
