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

// Timesteps per forward/eligibility block: the eligibility traces are read
// and written once per block.  The workspace holds per-step vectors for this
// many steps, independent of the sequence length.
constexpr int kBlockSteps = 32;

struct Layer {
  int n_inl = 0, n_pre = 0;
  int ldj = 0;    // n_rec rounded to 4: row stride of per-neuron vectors and traces
  int lda = 0;    // n_adaptive rounded to 4: row stride of epsa
  int kout = 0;   // n_out rounded to 32: rows of deltaK
  int npad = 0;   // n_rec rounded to 32: rows of ztK
  int rows_per_wave = 0;
  const float* W_src = nullptr;
  const float* Wout_src = nullptr;
  float *Wt, *Wop;                       // packed weights
  float *v, *a, *ztil, *zbar, *y;        // neuron, filter and readout state
  uint8_t* z;                            // spikes of the last step
  double* lossacc;                       // [B]
  float *psiK, *LK, *zbarK, *deltaK, *ztK, *Cpart;   // per-block vectors
  double *acc, *accout;                  // gradient accumulators
  float *ebar, *epsa;                    // eligibility traces
};

struct Plan {
  eprop_config cfg;
  std::vector<Layer> layers;
  int* err_flag = nullptr;
  int Kmax = kBlockSteps, Bp = 0, ldbk = 0, jlist = 0, out_splits = 1;
  size_t smem = 0;
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
  if (c->n_out > 1024) { *why = "n_out must be <= 1024"; return false; }
  if (c->n_rec > 16384) { *why = "n_rec must be <= 16384"; return false; }
  if (c->n_in > 65536) { *why = "n_in must be <= 65536"; return false; }
  if (c->recurrent != 0 && c->recurrent != 1) { *why = "recurrent must be 0 or 1"; return false; }
  if (c->n_adaptive < 0 || c->n_adaptive > c->n_rec) {
    *why = "n_adaptive must be in [0, n_rec]";
    return false;
  }
  const float k[] = {c->alpha, c->rho, c->kappa, c->thr, c->beta, c->gamma};
  for (float v : k)
    if (!std::isfinite(v)) { *why = "constants must be finite"; return false; }
  if (!(c->thr > 0.0f)) { *why = "thr must be > 0"; return false; }
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
  const size_t B = c.batch, N = c.n_rec, K = c.n_out, KM = plan->Kmax;
  plan->Bp = (int)round_up(B, 16);
  plan->ldbk = (int)(KM * plan->Bp);
  plan->jlist = (int)round_up(N, eprop::kFwdThreads) / eprop::kFwdThreads * 64;
  {
    int dummy;
    choose_splits(c.n_out, c.n_rec, plan->ldbk, 16, &plan->out_splits, &dummy);
  }
  plan->err_flag = (int*)take(sizeof(int));
  int rwmax = 0;
  for (int l = 0; l < c.n_layers; ++l) {
    Layer& L = plan->layers[l];
    L.n_inl = (l == 0) ? c.n_in : c.n_rec;
    L.n_pre = L.n_inl + (c.recurrent ? c.n_rec : 0);
    L.ldj = (int)round_up(N, 4);
    L.lda = (int)round_up(std::max(c.n_adaptive, 1), 4);
    L.kout = (int)round_up(K, 32);
    L.npad = (int)round_up(N, 32);
    L.rows_per_wave = (int)round_up((L.n_pre + 3) / 4, 64);
    rwmax = std::max(rwmax, L.rows_per_wave);
    const size_t np = L.n_pre;
    L.Wt = (float*)take(sizeof(float) * np * L.ldj);
    L.Wop = (float*)take(sizeof(float) * K * L.ldj);
    L.v = (float*)take(sizeof(float) * B * N);
    L.a = (float*)take(sizeof(float) * B * N);
    L.ztil = (float*)take(sizeof(float) * B * N);
    L.zbar = (float*)take(sizeof(float) * B * np);
    L.y = (float*)take(sizeof(float) * B * K);
    L.z = (uint8_t*)take(B * N);
    L.lossacc = (double*)take(sizeof(double) * B);
    L.psiK = (float*)take(sizeof(float) * B * KM * L.ldj);
    L.LK = (float*)take(sizeof(float) * B * KM * L.ldj);
    L.zbarK = (float*)take(sizeof(float) * np * B * KM);
    L.deltaK = (float*)take(sizeof(float) * L.kout * plan->ldbk);
    L.ztK = (float*)take(sizeof(float) * L.npad * plan->ldbk);
    L.Cpart = (float*)take(sizeof(float) * plan->out_splits * K * N);
    L.acc = (double*)take(sizeof(double) * np * L.ldj);
    L.accout = (double*)take(sizeof(double) * K * L.ldj);
    L.ebar = (float*)take(sizeof(float) * B * np * L.ldj);
    L.epsa = (float*)take(c.n_adaptive > 0 ? sizeof(float) * B * np * L.lda : 0);
  }
  const size_t npad4 = round_up(N, 4);
  plan->smem = sizeof(int) * (4 * (size_t)rwmax + 4 * (size_t)plan->jlist + 8) +
               sizeof(float) * (2 * K + 2) + (size_t)c.n_layers * 2 * npad4;
  plan->bytes = round_up(off, 256);
}

bool plan_fits(const Plan& p, std::string* why) {
  if (p.smem > 64 * 1024) {
    *why = "shape needs more than 64 KiB of shared memory in the forward kernel";
    return false;
  }
  return true;
}

}  // namespace

struct eprop_ctx {
  Plan plan;
  char* ws = nullptr;
  size_t ws_bytes = 0;
  hipStream_t stream = nullptr;
  long long t = 0;      // steps since the last reset
  int last_steps = 1;   // steps of the last block (where the last step's vectors sit)
  bool alive = false;
  std::string err;
  // profiling of the eligibility kernel
  bool prof = false;
  std::vector<hipEvent_t> ev;
  std::vector<int> prof_steps;
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
  const eprop_config& c = ctx->plan.cfg;
  for (Layer& L : ctx->plan.layers) {
    // drive weights transposed: Wt[i][j] = W[j][i], rows contiguous over j
    int rc = check(ctx, eprop::launch_pack(L.W_src, c.n_rec, L.n_pre, L.Wt, L.ldj, L.n_pre, 1,
                                           ctx->stream), "weight packing");
    if (rc) return rc;
    rc = check(ctx, eprop::launch_pack(L.Wout_src, c.n_out, c.n_rec, L.Wop, L.ldj, c.n_out, 0,
                                       ctx->stream), "readout weight packing");
    if (rc) return rc;
  }
  return EPROP_OK;
}

// Zeroes the neuron, filter and readout state.  Traces and accumulators are
// not cleared: the first block after a reset treats them as zero without
// reading them.
int clear_state(eprop_ctx* ctx) {
  const eprop_config& c = ctx->plan.cfg;
  const size_t B = c.batch, N = c.n_rec, K = c.n_out;
  hipStream_t s = ctx->stream;
  int rc = check(ctx, hipMemsetAsync(ctx->plan.err_flag, 0, sizeof(int), s), "reset");
  for (Layer& L : ctx->plan.layers) {
    if (rc) return rc;
    hipError_t e = hipSuccess;
    e = e ? e : hipMemsetAsync(L.v, 0, sizeof(float) * B * N, s);
    e = e ? e : hipMemsetAsync(L.a, 0, sizeof(float) * B * N, s);
    e = e ? e : hipMemsetAsync(L.ztil, 0, sizeof(float) * B * N, s);
    e = e ? e : hipMemsetAsync(L.zbar, 0, sizeof(float) * B * L.n_pre, s);
    e = e ? e : hipMemsetAsync(L.y, 0, sizeof(float) * B * K, s);
    e = e ? e : hipMemsetAsync(L.z, 0, B * N, s);
    e = e ? e : hipMemsetAsync(L.lossacc, 0, sizeof(double) * B, s);
    rc = check(ctx, e, "reset");
  }
  ctx->t = 0;
  return rc;
}

// `steps` (1..Kmax) consecutive timesteps: forward of every layer, readout
// gradient, eligibility traces and gradient accumulation.
int do_block(eprop_ctx* ctx, const uint8_t* x, int steps, const int32_t* labels, uint32_t* spikes) {
  const Plan& P = ctx->plan;
  const eprop_config& c = P.cfg;
  hipStream_t s = ctx->stream;
  const int first = ctx->t == 0;
  int rc;

  eprop::FwdArgs fa;
  for (int l = 0; l < 2; ++l) {
    eprop::FwdLayer& f = fa.L[l];
    if (l >= c.n_layers) { f = fa.L[0]; continue; }
    const Layer& L = P.layers[l];
    f.Wt = L.Wt; f.ldw = L.ldj; f.Wout = L.Wop; f.ldo = L.ldj;
    f.v = L.v; f.a = L.a; f.ztil = L.ztil; f.z = L.z; f.zbar = L.zbar; f.y = L.y;
    f.lossacc = L.lossacc; f.psiK = L.psiK; f.LK = L.LK; f.zbarK = L.zbarK;
    f.deltaK = L.deltaK; f.ztK = L.ztK;
    f.n_inl = L.n_inl; f.n_pre = L.n_pre; f.rows_per_wave = L.rows_per_wave;
  }
  fa.n_layers = c.n_layers; fa.x = x; fa.n_in = c.n_in; fa.labels = labels;
  fa.err_flag = P.err_flag; fa.spikes = spikes; fa.W32 = (c.n_rec + 31) / 32;
  fa.B = c.batch; fa.Bp = P.Bp; fa.n_rec = c.n_rec; fa.K_out = c.n_out;
  fa.n_adaptive = c.n_adaptive; fa.Kmax = P.Kmax; fa.steps = steps;
  fa.ldj = P.layers[0].ldj; fa.ldbk = P.ldbk; fa.jlist = P.jlist;
  fa.alpha = c.alpha; fa.rho = c.rho; fa.kappa = c.kappa; fa.thr = c.thr; fa.beta = c.beta;
  fa.gamma_over_thr = c.gamma / c.thr; fa.smem = P.smem;
  if ((rc = check(ctx, eprop::launch_forward(fa, s), "forward kernel"))) return rc;

  for (int l = 0; l < c.n_layers; ++l) {
    const Layer& L = P.layers[l];
    // dW_out += sum over (t, b) of delta (x) ztilde: MFMA GEMM, then fp64 accumulation
    eprop::GemmArgs g;
    g.A = L.deltaK; g.Bm = L.ztK; g.C = L.Cpart;
    g.M = c.n_out; g.N = c.n_rec; g.K = steps * P.Bp; g.lda = P.ldbk; g.ldb = P.ldbk;
    g.ldc = c.n_rec;
    choose_splits(g.M, g.N, g.K, P.out_splits, &g.splits, &g.k_chunk);
    g.split_stride = (size_t)c.n_out * c.n_rec;
    if ((rc = check(ctx, eprop::launch_gemm_nt(g, s), "readout gradient GEMM"))) return rc;
    if ((rc = check(ctx, eprop::launch_accumulate(L.Cpart, g.splits, g.split_stride, c.n_out,
                                                  c.n_rec, L.accout, L.ldj, first, s),
                    "readout gradient accumulation")))
      return rc;

    eprop::TraceArgs ta;
    ta.ebar = L.ebar; ta.epsa = L.epsa; ta.acc = L.acc; ta.zbarK = L.zbarK;
    ta.psiK = L.psiK; ta.LK = L.LK; ta.B = c.batch; ta.n_pre = L.n_pre; ta.n_post = c.n_rec;
    ta.ldj = L.ldj; ta.n_adaptive = c.n_adaptive; ta.lda = L.lda; ta.Kmax = P.Kmax;
    ta.steps = steps; ta.kappa = c.kappa; ta.rho = c.rho; ta.beta = c.beta; ta.first = first;
    const bool timed = ctx->prof && ctx->prof_n < ctx->prof_max;
    if (timed && (rc = check(ctx, hipEventRecord(ctx->ev[2 * ctx->prof_n], s), "event record")))
      return rc;
    if ((rc = check(ctx, eprop::launch_trace(ta, s), "eligibility kernel"))) return rc;
    if (timed) {
      if ((rc = check(ctx, hipEventRecord(ctx->ev[2 * ctx->prof_n + 1], s), "event record")))
        return rc;
      ctx->prof_steps[ctx->prof_n] = steps;
      ctx->prof_n++;
    }
  }
  ctx->t += steps;
  ctx->last_steps = steps;
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
  if (!plan_fits(p, &why)) {
    g_last_error = why;
    return 0;
  }
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
  if (!plan_fits(probe, &why)) return fail(nullptr, EPROP_EINVAL, why);
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
  return do_block(ctx, d_x_t, 1, d_labels, d_spikes_t);
}

int eprop_run_sequence(eprop_ctx* ctx, const uint8_t* d_x, int32_t T, const int32_t* d_labels,
                       uint32_t* d_spikes) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (!d_x || !d_labels) return fail(ctx, EPROP_EINVAL, "x or labels is NULL");
  if (T < 1) return fail(ctx, EPROP_EINVAL, "T must be >= 1");
  const eprop_config& c = ctx->plan.cfg;
  const size_t x_step = (size_t)c.batch * c.n_in;
  const size_t s_step = (size_t)c.n_layers * c.batch * ((c.n_rec + 31) / 32);
  for (int32_t t = 0; t < T;) {
    const int steps = std::min<int32_t>(ctx->plan.Kmax, T - t);
    int rc = do_block(ctx, d_x + t * x_step, steps, d_labels,
                      d_spikes ? d_spikes + t * s_step : nullptr);
    if (rc) return rc;
    t += steps;
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
  ctx->prof_steps.assign(max_launches, 0);
  return EPROP_OK;
}

int eprop_profile_end(eprop_ctx* ctx, double* total_ms, int32_t* n_launches, int64_t* n_steps) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (!total_ms || !n_launches || !n_steps) return fail(ctx, EPROP_EINVAL, "output pointer is NULL");
  int rc = check(ctx, hipStreamSynchronize(ctx->stream), "stream synchronize");
  if (rc) return rc;
  double sum = 0.0;
  for (int k = 0; k < ctx->prof_n; ++k) {
    float ms = 0.0f;
    rc = check(ctx, hipEventElapsedTime(&ms, ctx->ev[2 * k], ctx->ev[2 * k + 1]), "event time");
    if (rc) return rc;
    sum += ms;
  }
  int64_t steps = 0;
  for (int k = 0; k < ctx->prof_n; ++k) steps += ctx->prof_steps[k];
  *total_ms = sum;
  *n_launches = ctx->prof_n;
  *n_steps = steps;
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
  const int64_t kstride = (int64_t)ctx->plan.Kmax * L.ldj;   // rows of psiK, LK are [b][t]
  const int64_t tl = ctx->last_steps - 1;
  switch (which) {
    case 0: *d_ptr = L.v; *cols = c.n_rec; *ld = c.n_rec; break;
    case 1: *d_ptr = L.a; *cols = c.n_rec; *ld = c.n_rec; break;
    case 2: *d_ptr = L.psiK + tl * L.ldj; *cols = c.n_rec; *ld = kstride; break;
    case 3: *d_ptr = L.LK + tl * L.ldj; *cols = c.n_rec; *ld = kstride; break;
    case 4: *d_ptr = L.y; *cols = c.n_out; *ld = c.n_out; break;
    default: return fail(ctx, EPROP_EINVAL, "unknown buffer");
  }
  return EPROP_OK;
}

}  // extern "C"
