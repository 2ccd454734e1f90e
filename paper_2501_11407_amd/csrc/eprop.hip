// Host side of the e-prop library: C ABI (include/eprop.h), workspace
// layout and the per-step launch schedule.  No device memory is allocated
// here: every buffer is carved from the caller's workspace.
#include "../../include/eprop.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"

namespace {

thread_local std::string g_last_error = "";

size_t round_up(size_t v, size_t m) { return (v + m - 1) / m * m; }

// Split-K choice for a GEMM of M x N over K (multiple of 16): about 4096
// waves (four per SIMD: the k loop is latency-bound), at most max_splits,
// chunks a multiple of 16.
constexpr int kMaxOutSplits = 64;
void choose_splits(int M, int N, int K, int max_splits, int* splits, int* k_chunk) {
  const long long tiles = (long long)((M + 31) / 32) * ((N + 31) / 32);
  long long want = std::max<long long>(1, (4096 + tiles - 1) / tiles);
  want = std::min<long long>(want, std::max(1, K / 16));
  want = std::min<long long>(want, max_splits);
  int kc = (int)round_up((K + want - 1) / want, 16);
  kc = std::max(kc, 16);
  *k_chunk = kc;
  *splits = (K + kc - 1) / kc;
}

// Timesteps per forward/eligibility block (eprop::kBlockSteps): the
// eligibility traces are read and written once per block, and the block's
// contractions over its steps run on the matrix cores.  The workspace holds
// per-step vectors for this many steps, independent of the sequence length.
using eprop::kBlockSteps;

// Per-block buffers rotate through the plan's slots (kSlots, or one on a
// single stream): the forward of block k may start once the eligibility pass
// of block k - kSlots has released its slot.  With three, the forward, the
// passes between it and the eligibility kernel, and the eligibility kernel
// of three consecutive blocks run at once, and a block costs the longest of
// the three rather than the sum of two of them.
constexpr int kSlots = 3;

struct Layer {
  int n_inl = 0, n_pre = 0;
  int n_pre_pad = 0;   // n_pre rounded to the eligibility kernel's row group
  int ldj = 0;    // n_rec rounded to 4: row stride of traces and accumulators
  int ldv = 0;    // n_rec rounded to 256: row stride of psiK, LK
  int ldw = 0;    // 512 QN (forward positions): row stride of Wt
  int16_t* W16 = nullptr;   // the drive weights times 2^14 as int16 (FwdLayer::W16)
  const float* W_src = nullptr;
  const float* Wout_src = nullptr;
  const float* Fb_src = nullptr;         // feedback matrix of the learning signal (NULL: W_out)
  float *Wt, *WoutT, *FbT;               // packed weights
  float *v, *a, *ztil, *zbar, *y;        // neuron, filter and readout state
  uint8_t* z;                            // spikes of the last step
  double* lossacc;                       // [B]
  // per-block vectors in up to kSlots slots: the forward of block k+1 fills one
  // while the eligibility pass of block k reads another
  float *psiK[kSlots], *LK[kSlots], *deltaK[kSlots], *ztK[kSlots];
  // the binary presynaptic values (one bit per row and step, a 16-bit word
  // per row and 16-step chunk), and the block
  // coefficients of the eligibility recursion as scaled fp16 pairs
  uint16_t* pbits[kSlots];
  uint32_t* coefO[kSlots];        // the coefficient operands, tile-major (OpLayout)
  float* coefS[kSlots];
  float* zstart[kSlots];                 // presynaptic filter at each block's start [B][ldi]
  float* Cpart;
  double *acc, *accout;                  // gradient accumulators (acc: n_split partials)
  int n_split = 1;                       // batch splits of the eligibility kernel
  size_t acc_stride = 0;                 // doubles between partial accumulators
  float *ebar, *epsa;                    // eligibility traces
  float* epsv = nullptr;                 // reset_grad: per-synapse membrane eligibility
};

// A neuron step linear in its state: h = A h_prev + b I + r z_prev, spike
// argument c . h - thr (see derive_neuron).
struct NeuronCoef {
  double A[2][2], b[2], r[2], c[2];
};

// At most two layers, held in place (a plan allocates nothing).
struct Layers {
  Layer l[2];
  int n = 0;
  void assign(int count, const Layer& v) {
    n = count;
    for (int k = 0; k < 2; ++k) l[k] = v;
  }
  Layer& operator[](int k) { return l[k]; }
  const Layer& operator[](int k) const { return l[k]; }
  Layer* begin() { return l; }
  Layer* end() { return l + n; }
  const Layer* begin() const { return l; }
  const Layer* end() const { return l + n; }
};

struct Plan {
  eprop_config cfg;
  Layers layers;
  // three-trace recursion (reset path kept, or the two-compartment neuron),
  // and the neurons whose second state component has per-synapse traces
  int rt = 0, na2 = 0;
  eprop::OpLayout ol{};             // coefficient operands, tile-major
  int slots = kSlots;               // per-block buffer sets in use
  NeuronCoef gen{};                 // two-compartment neuron: derived step
  int* err_flag = nullptr;
  int* w16ok = nullptr;             // [2]: the int16 drive weights are exact, their largest |k| (launch_pack16)
  // the first layer's input drive of a block and its active-input counts
  // (launch_input_drive), in two buffers: the next block's may be computed
  // while the forward of the current one reads the other
  float* Iin[2] = {};
  int* nin[2] = {};
  int Kmax = kBlockSteps, Bp = 0, rows = 0, ldk = 0, ldn = 0, ldc = 0, jlist = 0, out_splits = 1;
  size_t smem = 0;
  int svc = 0;                      // the forward's service wave (FwdArgs::svc)
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
  // the forward keeps at most 16 neurons per thread of its 512
  if (c->n_rec > 16 * eprop::kFwdThreads) { *why = "n_rec must be <= 8192"; return false; }
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
  if (!(c->alpha >= 0.0f && c->alpha < 1.0f)) {
    *why = "alpha must be in [0, 1) (the presynaptic filter must be bounded)";
    return false;
  }
  if (c->reset_grad != 0 && c->reset_grad != 1) { *why = "reset_grad must be 0 or 1"; return false; }
  if (c->neuron_model != 0 && c->neuron_model != 1) { *why = "neuron_model must be 0 or 1"; return false; }
  if (c->neuron_model == 1) {
    if (c->n_adaptive != 0) { *why = "the two-compartment neuron has no adaptive threshold (n_adaptive 0)"; return false; }
    const float k2[] = {c->alpha_d, c->coupling, c->bap};
    for (float v : k2)
      if (!std::isfinite(v)) { *why = "constants must be finite"; return false; }
  }
  return true;
}

// ---------------------------------------------------------------- neuron models
// Forward-mode dual numbers: a value and its derivative along one direction.
struct Dual {
  double v = 0.0, d = 0.0;
};
Dual operator+(Dual a, Dual b) { return {a.v + b.v, a.d + b.d}; }
Dual operator-(Dual a, Dual b) { return {a.v - b.v, a.d - b.d}; }
Dual operator*(Dual a, Dual b) { return {a.v * b.v, a.d * b.v + a.v * b.d}; }
Dual konst(double x) { return {x, 0.0}; }

// The neuron models' step over a scalar type T, as the forward kernel and
// the paper's Eq. (8) write them: state h (component 0: the membrane or soma,
// the one the reset acts on), drive I, last spike zp -> new state, and the
// spike argument u(h) (spike iff u > 0).  cls 1: adaptive neurons.
template <typename T>
void model_step(const eprop_config& c, int cls, const T (&h)[2], T I, T zp, T (&out)[2]) {
  const T thr = konst(c.thr);
  if (c.neuron_model == 1) {   // soma s = h0, dendrite d = h1
    out[1] = konst(c.alpha_d) * h[1] + I + konst(c.bap) * zp;
    out[0] = konst(c.alpha) * h[0] + konst(c.coupling) * h[1] - thr * zp;
  } else {                     // membrane v = h0, adaptation a = h1
    out[0] = konst(c.alpha) * h[0] + I - thr * zp;
    out[1] = konst(c.rho) * h[1] + zp;
  }
}
template <typename T>
T model_arg(const eprop_config& c, int cls, const T (&h)[2]) {
  if (c.neuron_model == 1) return h[0] - konst(c.thr);
  const double beta = cls == 1 ? c.beta : 0.0;
  return h[0] - (konst(c.thr) + konst(beta) * h[1]);
}

// Coefficients of a step that is linear in (h, I, zp): A = dh/dh_prev,
// b = dh/dI, r = dh/dzp (the own-spike paths; the reset of component 0 is
// gradient-stopped unless reset_grad), c = du/dh, each column one dual pass.
// The derivatives are taken at two different points and must agree (else
// the step is not linear and the block form does not apply).
bool derive_neuron(const eprop_config& cfg, int cls, NeuronCoef* out) {
  const double pts[2][4] = {{0.3, -0.2, 0.7, 1.0}, {-1.1, 0.45, -0.3, 0.0}};
  NeuronCoef k[2];
  for (int p = 0; p < 2; ++p) {
    for (int dir = 0; dir < 4; ++dir) {   // h0, h1, I, zp
      Dual h[2] = {{pts[p][0], dir == 0 ? 1.0 : 0.0}, {pts[p][1], dir == 1 ? 1.0 : 0.0}};
      Dual I{pts[p][2], dir == 2 ? 1.0 : 0.0}, zp{pts[p][3], dir == 3 ? 1.0 : 0.0};
      Dual o[2];
      model_step(cfg, cls, h, I, zp, o);
      for (int m = 0; m < 2; ++m) {
        if (dir < 2) k[p].A[m][dir] = o[m].d;
        else if (dir == 2) k[p].b[m] = o[m].d;
        else k[p].r[m] = o[m].d;
      }
    }
    for (int dir = 0; dir < 2; ++dir) {
      Dual h[2] = {{pts[p][0], dir == 0 ? 1.0 : 0.0}, {pts[p][1], dir == 1 ? 1.0 : 0.0}};
      k[p].c[dir] = model_arg(cfg, cls, h).d;
    }
  }
  // the same derivatives at both points (== treats the two zeros as one)
  const double* k0 = &k[0].A[0][0];
  const double* k1 = &k[1].A[0][0];
  constexpr int nk = sizeof(NeuronCoef) / sizeof(double);
  for (int q = 0; q < nk; ++q)
    if (!(k0[q] == k1[q])) return false;
  *out = k[0];
  double* o = &out->A[0][0];
  for (int q = 0; q < nk; ++q) o[q] = o[q] + 0.0;   // -0 -> +0
  if (!cfg.reset_grad) out->r[0] = 0.0;   // the reset stays gradient-stopped
  return true;
}

// Lays the workspace out (base == nullptr: sizing only) with `slots` sets of
// per-block buffers.
void make_plan(const eprop_config& c, char* base, Plan* plan, int slots = kSlots) {
  plan->cfg = c;
  plan->slots = slots;
  plan->layers.assign(c.n_layers, Layer());
  plan->rt = (c.reset_grad || c.neuron_model == 1) ? 1 : 0;
  plan->na2 = c.neuron_model == 1 ? c.n_rec : c.n_adaptive;
  if (c.neuron_model == 1) derive_neuron(c, 0, &plan->gen);
  size_t off = 0;
  auto take = [&](size_t bytes) -> char* {
    off = round_up(off, 256);
    char* p = base ? base + off : nullptr;
    off += round_up(std::max<size_t>(bytes, 1), 256);
    return p;
  };
  const size_t B = c.batch, N = c.n_rec, K = c.n_out, KM = plan->Kmax;
  plan->Bp = (int)round_up(B, 16);
  plan->rows = (int)round_up(KM * plan->Bp, 32);     // rows of deltaK, ztK, psiK, LK
  plan->ldk = (int)round_up(K, 32);
  plan->ldn = (int)round_up(N, 32);
  plan->ldc = (int)round_up(N, eprop::kColPad);
  {
    const int n_jt = (int)((N + eprop::kTileJ - 1) / eprop::kTileJ);
    plan->ol.n_jt_a = (plan->na2 + eprop::kTileJ - 1) / eprop::kTileJ;
    plan->ol.nxa = 3 + plan->rt;      // U, H, V (, W)
    plan->ol.nxl = 2 + plan->rt;      // U, H (, W)
    plan->ol.cw = 256 * (plan->ol.n_jt_a * plan->ol.nxa + (n_jt - plan->ol.n_jt_a) * plan->ol.nxl);
  }
  const int qn = eprop::forward_qn((int)N);
  plan->jlist = qn * 64;   // a wave's neurons
  {
    int dummy;
    choose_splits(c.n_out, c.n_rec, (int)(KM * plan->Bp), kMaxOutSplits, &plan->out_splits, &dummy);
  }
  const size_t R = plan->rows;
  plan->err_flag = (int*)take(sizeof(int));
  plan->w16ok = (int*)take(2 * sizeof(int));
  for (int l = 0; l < c.n_layers; ++l) {
    Layer& L = plan->layers[l];
    L.n_inl = (l == 0) ? c.n_in : c.n_rec;
    L.n_pre = L.n_inl + (c.recurrent ? c.n_rec : 0);
    L.n_pre_pad = (int)round_up(L.n_pre, eprop::kRowPad);
    L.ldj = (int)round_up(N, 4);
    L.ldv = (int)round_up(N, 256);
    L.ldw = qn * eprop::kFwdThreads;
    const size_t np = L.n_pre, npp = L.n_pre_pad;
    // one more row each, of zeros: the forward's drive loads of a batch's
    // entries past the active list read it
    L.Wt = (float*)take(sizeof(float) * (np + 1) * L.ldw);
    L.W16 = (int16_t*)take(sizeof(int16_t) * (np + 1) * L.ldw);
    L.WoutT = (float*)take(sizeof(float) * plan->ldn * plan->ldk);
    L.FbT = (float*)take(sizeof(float) * plan->ldn * plan->ldk);
    L.v = (float*)take(sizeof(float) * B * N);
    L.a = (float*)take(sizeof(float) * B * N);
    L.ztil = (float*)take(sizeof(float) * B * N);
    L.zbar = (float*)take(sizeof(float) * B * np);
    L.y = (float*)take(sizeof(float) * B * K);
    L.z = (uint8_t*)take(B * N);
    L.lossacc = (double*)take(sizeof(double) * B);
    for (int sl = 0; sl < slots; ++sl) {
      L.psiK[sl] = (float*)take(sizeof(float) * R * L.ldv);
      L.LK[sl] = (float*)take(sizeof(float) * R * L.ldv);
      L.deltaK[sl] = (float*)take(sizeof(float) * R * plan->ldk);
      L.ztK[sl] = (float*)take(sizeof(float) * R * plan->ldn);
    }
    L.Cpart = (float*)take(sizeof(float) * plan->out_splits * K * N);
    // batch splits of the eligibility kernel: about 2048 workgroups (four
    // rounds of two per compute unit; at most 8 splits for that), and enough
    // splits that a workgroup walks at most about 26 batch elements (the row
    // tiles that share a coefficient chunk drift apart in L2 over longer
    // walks); at most 32, one per element, and 2 GiB of fp64 partials
    const size_t tiles = (npp / eprop::kTileI) * ((N + eprop::kTileJ - 1) / eprop::kTileJ);
    L.acc_stride = npp * L.ldj;
    const size_t by_tiles = std::min<size_t>(8, (2048 + tiles - 1) / tiles);
    const size_t by_batch = (B + 25) / 26;
    const size_t by_memory = std::max<size_t>(1, ((size_t)2 << 30) / (sizeof(double) * L.acc_stride));
    L.n_split = (int)std::max<size_t>(
        1, std::min<size_t>({std::max(by_tiles, by_batch), 32, B, by_memory}));
    L.acc = (double*)take(sizeof(double) * L.n_split * L.acc_stride);
    L.accout = (double*)take(sizeof(double) * K * L.ldj);
    // traces tile by tile: all j tiles, and the tiles holding adaptive neurons
    const size_t ldc = round_up(N, eprop::kColPad);
    const size_t lda_t = round_up(plan->na2, eprop::kTileJ);
    L.ebar = (float*)take(sizeof(float) * B * npp * ldc);
    L.epsa = (float*)take(plan->na2 > 0 ? sizeof(float) * B * npp * lda_t : 0);
    // with the reset path kept (or two compartments), the first state
    // component's eligibility per synapse as well
    L.epsv = plan->rt ? (float*)take(sizeof(float) * B * npp * ldc) : nullptr;
  }
  for (int k = 0; k < 2; ++k) {
    plan->Iin[k] = (float*)take(sizeof(float) * KM * B * qn * eprop::kFwdThreads);
    plan->nin[k] = (int*)take(sizeof(int) * KM * B);
  }
  for (Layer& L : plan->layers) {
    const size_t ldc = plan->ldc;
    for (int sl = 0; sl < slots; ++sl) {
      // p: one bit per row and step (a 16-bit word per row and 16-step
      // chunk); coefficients: a scaled fp16 pair per value (4 bytes)
      L.pbits[sl] = (uint16_t*)take(sizeof(uint16_t) * B * L.n_pre_pad * (KM / eprop::kChunk));
      L.coefO[sl] = (uint32_t*)take(sizeof(uint32_t) * B * (KM / eprop::kChunk) * plan->ol.cw);
      const int planes = plan->rt ? eprop::kScalarPlanesRT : eprop::kScalarPlanes;
      L.coefS[sl] = (float*)take(sizeof(float) * planes * B * ldc);
    }
    for (int sl = 0; sl < slots; ++sl) L.zstart[sl] = (float*)take(sizeof(float) * B * L.n_pre_pad);
  }
  // the forward's shared memory (FwdLds): spike lists and their lengths by
  // step parity, the block's input counts, readout partial sums and outputs
  // (the filter of the rows and the spikes are in registers)
  const size_t NL = c.n_layers, W = eprop::kFwdWaves;
  const size_t smem_base = sizeof(int) * (NL * 2 * W * plan->jlist + NL * 2 * W + KM) +
                           sizeof(float) * (NL * 2 * W * K + NL * K);
  // the forward's service wave and its input-drive ring (three steps of 512
  // QN floats) where that fits beside an eligibility workgroup
  const size_t ring = (size_t)3 * qn * eprop::kFwdThreads * sizeof(float);
  const size_t fwd_smem = smem_base;
  // with up to two neurons per thread: with more, the ninth wave's third
  // wave on one SIMD would keep every eligibility workgroup off the forward's
  // compute units (registers); measured on two layers of 2048 neurons, the
  // forward without it lets the eligibility passes run beside it, 4% faster
  plan->svc = qn <= 2;
  plan->smem = fwd_smem + (plan->svc ? ring : 0);
  plan->bytes = round_up(off, 256);
}

bool plan_fits(const Plan& p, std::string* why) {
  if (p.smem > 160 * 1024) {
    *why = "shape needs more than 160 KiB of shared memory in the forward kernel";
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
  int slot = 0;         // K-buffer slot the next block writes
  int last_slot = 0;    // slot of the last block
  bool slot_used[kSlots] = {};
  // internal streams: the forward kernel, and the passes between it and the
  // eligibility kernel (learning signal, readout gradient, coefficients)
  hipStream_t fwd_stream = nullptr, coef_stream = nullptr;
  hipEvent_t ev_entry = nullptr, ev_fwd[kSlots] = {}, ev_coef[kSlots] = {}, ev_out[kSlots] = {},
            ev_done[kSlots] = {};
  // every kernel on the caller's stream, in issue order, with no streams or
  // events of the context's own (the entry point that allocates nothing)
  bool single_stream = false;
  // online weight application (eprop_set_online): every `online_every` steps
  // since the reset, before the next step runs
  float online_lr = 0.0f;
  int online_every = 0;
  int split_mode = EPROP_SPLIT_AUTO;   // eprop_set_block_split
  long long online_applied = -1;   // step count of the last update
  hipEvent_t ev_update = nullptr;
  // the first layer's input drive of the next block of a sequence, computed
  // on in_stream while the forward of the current block runs: ev_pre is
  // recorded on the forward stream before that forward (the weights, the
  // inputs and the other buffer are then ready), ev_in[k] when buffer k is
  // filled; in_buf is the buffer the next block reads, in_ready whether it
  // has been filled for it
  hipStream_t in_stream = nullptr;
  hipEvent_t ev_pre = nullptr, ev_in[2] = {};
  int in_buf = 0;
  bool in_ready = false;
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
  // the int16 drive weights are used when every layer's are exact
  int rc0 = check(ctx, eprop::launch_set_flag(ctx->plan.w16ok, 1, ctx->stream), "weight packing");
  if (rc0) return rc0;
  // the row of zeros after each layer's drive rows (row n_pre of W16 and Wt),
  // read by the forward's loads past a step's active list
  eprop::ZeroRanges zr{};
  for (Layer& L : ctx->plan.layers) {
    zr.p[zr.n] = L.W16 + (size_t)L.n_pre * L.ldw;
    zr.bytes[zr.n++] = sizeof(int16_t) * L.ldw;
    zr.p[zr.n] = L.Wt + (size_t)L.n_pre * L.ldw;
    zr.bytes[zr.n++] = sizeof(float) * L.ldw;
  }
  rc0 = check(ctx, eprop::launch_zero_many(zr, ctx->stream), "weight packing");
  if (rc0) return rc0;
  for (Layer& L : ctx->plan.layers) {
    int rc16 = check(ctx, eprop::launch_pack16(L.W_src, c.n_rec, L.n_pre, L.W16,
                                               eprop::forward_qn(c.n_rec), ctx->plan.w16ok,
                                               ctx->stream), "weight packing");
    if (rc16) return rc16;
    // drive weights transposed, Wt[i][j] = W[j][i], columns padded to the
    // forward workgroup size
    int rc = check(ctx, eprop::launch_pack(L.W_src, c.n_rec, L.n_pre, L.Wt, L.ldw, L.n_pre, 1,
                                           ctx->stream), "weight packing");
    if (rc) return rc;
    // WoutT[j][k] = Wout[k][j]: the readout, and the B operand of the
    // learning-signal GEMM unless a feedback matrix is set (packed the same way)
    rc = check(ctx, eprop::launch_pack(L.Wout_src, c.n_out, c.n_rec, L.WoutT, ctx->plan.ldk,
                                       ctx->plan.ldn, 1, ctx->stream), "readout weight packing");
    if (rc) return rc;
  }
  return EPROP_OK;
}

// FbT[j][k] = B[k][j] for every layer with a feedback matrix set; nothing
// else is rewritten (the weights in use stay what they are).
int pack_feedback(eprop_ctx* ctx) {
  const eprop_config& c = ctx->plan.cfg;
  for (Layer& L : ctx->plan.layers) {
    if (!L.Fb_src) continue;
    int rc = check(ctx, eprop::launch_pack(L.Fb_src, c.n_out, c.n_rec, L.FbT, ctx->plan.ldk,
                                           ctx->plan.ldn, 1, ctx->stream), "feedback matrix packing");
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
  // one fill kernel for every range rather than memset nodes, so that a
  // caller may capture it
  eprop::ZeroRanges zr{};
  auto add = [&](void* p, size_t bytes) {
    zr.p[zr.n] = p;
    zr.bytes[zr.n] = bytes;
    ++zr.n;
  };
  add(ctx->plan.err_flag, sizeof(int));
  for (Layer& L : ctx->plan.layers) {
    add(L.v, sizeof(float) * B * N);
    add(L.a, sizeof(float) * B * N);
    add(L.ztil, sizeof(float) * B * N);
    add(L.zbar, sizeof(float) * B * L.n_pre);
    add(L.y, sizeof(float) * B * K);
    add(L.z, B * N);
    add(L.lossacc, sizeof(double) * B);
  }
  static_assert(1 + 7 * 2 <= eprop::ZeroRanges::kMax, "ranges of two layers");
  int rc = check(ctx, eprop::launch_zero_many(zr, s), "reset");
  ctx->t = 0;
  ctx->online_applied = -1;
  return rc;
}

// The weights in use become W0 - lr * G on the 2^-14 grid (G: the gradient
// so far), on the caller's stream after the last eligibility pass; the next
// forward waits for it.
int apply_online(eprop_ctx* ctx) {
  const Plan& P = ctx->plan;
  const eprop_config& c = P.cfg;
  hipStream_t s = ctx->stream;
  int rc = check(ctx, eprop::launch_set_flag(P.w16ok, 1, s), "online weight update");
  for (int l = 0; l < c.n_layers && !rc; ++l) {
    const Layer& L = P.layers[l];
    eprop::OnlineArgs a;
    a.W0 = L.W_src; a.Wout0 = L.Wout_src;
    a.acc = L.acc; a.ldj = L.ldj; a.n_split = L.n_split; a.acc_stride = L.acc_stride;
    a.accout = L.accout; a.ld_acc = L.ldj;
    a.Wt = L.Wt; a.ldw = L.ldw; a.W16 = L.W16; a.qn = eprop::forward_qn(c.n_rec); a.ok = P.w16ok;
    a.WoutT = L.WoutT; a.ldk = P.ldk;
    a.n_rec = c.n_rec; a.n_pre = L.n_pre; a.n_inl = L.n_inl; a.recurrent = c.recurrent; a.K = c.n_out;
    a.lr = (double)ctx->online_lr;
    rc = check(ctx, eprop::launch_online_update(a, s), "online weight update");
  }
  if (ctx->single_stream) return rc;
  if (!rc) rc = check(ctx, hipEventRecord(ctx->ev_update, s), "event record");
  if (!rc) rc = check(ctx, hipStreamWaitEvent(ctx->fwd_stream, ctx->ev_update, 0), "stream wait");
  return rc;
}

// Rough costs that decide the block split, in microseconds on MI355X: one
// round trip of every layer's per-synapse traces through HBM at about half
// its peak bandwidth (the fixed part of an eligibility pass), and one
// timestep of the forward pass of every layer with the learning-signal and
// coefficient passes that follow it.
struct SplitCost {
  double round_trip_us = 0, step_us = 0;
};

SplitCost split_cost(const Plan& P) {
  const eprop_config& c = P.cfg;
  SplitCost k;
  const double per_syn = 1.0 + (double)P.na2 / c.n_rec + P.rt;   // traces per synapse
  for (const Layer& L : P.layers)
    k.round_trip_us += (double)c.batch * L.n_pre * c.n_rec * per_syn * 8.0 / 4.0e6;
  k.step_us = c.n_layers * (2.5 + (double)c.batch * c.n_rec * 32.0 / 4.0e6);
  return k;
}

// An online weight update falls before the step t steps after the reset.
bool online_due(const eprop_ctx* ctx, long long t) {
  return ctx->online_every > 0 && t > 0 && t % ctx->online_every == 0 && ctx->online_applied != t;
}

// `steps` (1..Kmax) consecutive timesteps: forward of every layer, readout
// gradient, eligibility traces and gradient accumulation.  x_next (NULL:
// none) and steps_next: the block that follows in the same call, whose
// input drive may be computed meanwhile.
int do_block(eprop_ctx* ctx, const uint8_t* x, int steps, const int32_t* labels, uint32_t* spikes,
             const uint8_t* x_next, int steps_next) {
  const Plan& P = ctx->plan;
  const eprop_config& c = P.cfg;
  hipStream_t s = ctx->stream;
  hipStream_t sf = ctx->fwd_stream;
  hipStream_t sc = ctx->coef_stream;
  const int first = ctx->t == 0;
  const int sl = ctx->slot;
  int rc;
  if (online_due(ctx, ctx->t)) {
    if ((rc = apply_online(ctx))) return rc;
    ctx->online_applied = ctx->t;
  }
  // The forward may overwrite this slot once the passes that read it
  // kSlots blocks ago are done.  (On one stream, issue order says so.)
  const bool ev = !ctx->single_stream;
  if (ev && ctx->slot_used[sl] &&
      (rc = check(ctx, hipStreamWaitEvent(sf, ctx->ev_done[sl], 0), "stream wait")))
    return rc;

  eprop::FwdArgs fa;
  for (int l = 0; l < 2; ++l) {
    eprop::FwdLayer& f = fa.L[l];
    const Layer& L = P.layers[std::min(l, c.n_layers - 1)];
    f.Wt = L.Wt; f.ldw = L.ldw; f.W16 = L.W16; f.WoutT = L.WoutT;
    f.v = L.v; f.a = L.a; f.ztil = L.ztil; f.z = L.z; f.zbar = L.zbar; f.y = L.y;
    f.lossacc = L.lossacc; f.psiK = L.psiK[sl]; f.pbits = L.pbits[sl]; f.zstart = L.zstart[sl];
    f.deltaK = L.deltaK[sl]; f.ztK = L.ztK[sl];
    f.n_inl = L.n_inl; f.n_pre = L.n_pre; f.ldi = L.n_pre_pad;
  }
  // the first layer's input rows: their drive before the forward (already
  // computed on the input stream, or now on the forward stream); their
  // filter and p bits on the coefficient stream (below)
  const Layer& L0 = P.layers[0];
  const int ib = ctx->in_buf;
  eprop::InputArgs ia;
  ia.x = x; ia.n_in = c.n_in; ia.B = c.batch; ia.steps = steps;
  ia.Wt = L0.Wt; ia.ldw = L0.ldw; ia.W16 = L0.W16; ia.qn = eprop::forward_qn(c.n_rec); ia.w16ok = P.w16ok;
  ia.Iin = P.Iin[ib]; ia.nin = P.nin[ib];
  ia.zbar = L0.zbar; ia.n_pre = L0.n_pre; ia.zstart = L0.zstart[sl]; ia.pbits = L0.pbits[sl];
  ia.ldi = L0.n_pre_pad; ia.alpha = c.alpha;
  if (ctx->in_ready) {
    ctx->in_ready = false;
    if ((rc = check(ctx, hipStreamWaitEvent(sf, ctx->ev_in[ib], 0), "stream wait"))) return rc;
  } else if ((rc = check(ctx, eprop::launch_input_drive(ia, sf), "input drive kernel"))) {
    return rc;
  }
  fa.Iin = P.Iin[ib]; fa.nin = P.nin[ib];
  fa.n_layers = c.n_layers; fa.labels = labels;
  fa.err_flag = P.err_flag; fa.w16ok = P.w16ok; fa.spikes = spikes; fa.W32 = (c.n_rec + 31) / 32;
  fa.B = c.batch; fa.Bp = P.Bp; fa.n_rec = c.n_rec; fa.K_out = c.n_out;
  fa.n_adaptive = c.n_adaptive; fa.Kmax = P.Kmax; fa.steps = steps;
  fa.ldj = P.layers[0].ldv; fa.ldk = P.ldk; fa.ldn = P.ldn; fa.jlist = P.jlist;
  fa.alpha = c.alpha; fa.rho = c.rho; fa.kappa = c.kappa; fa.thr = c.thr; fa.beta = c.beta;
  fa.gamma_over_thr = c.gamma / c.thr; fa.inv_thr = 1.0f / c.thr; fa.smem = P.smem; fa.svc = P.svc;
  fa.model = c.neuron_model;
  for (int m = 0; m < 2; ++m) {
    fa.mA[m][0] = (float)P.gen.A[m][0]; fa.mA[m][1] = (float)P.gen.A[m][1];
    fa.mb[m] = (float)P.gen.b[m]; fa.mc[m] = (float)P.gen.c[m];
  }
  // the forward uses the full own-spike terms (the reset included)
  {
    NeuronCoef full{};
    if (c.neuron_model == 1) {
      eprop_config cf = c;
      cf.reset_grad = 1;
      derive_neuron(cf, 0, &full);
    }
    fa.mr[0] = (float)full.r[0]; fa.mr[1] = (float)full.r[1];
  }
  // the next block's input drive into the other buffer, while this forward
  // runs (not when the weights change before the next block): the event that
  // lets it start is recorded before the forward, whose launch comes first
  // so that it does not wait for the host
  const bool pre = ev && x_next && steps_next > 0 && !online_due(ctx, ctx->t + steps);
  if (pre && (rc = check(ctx, hipEventRecord(ctx->ev_pre, sf), "event record"))) return rc;
  if ((rc = check(ctx, eprop::launch_forward(fa, sf), "forward kernel"))) return rc;
  if (ev && (rc = check(ctx, hipEventRecord(ctx->ev_fwd[sl], sf), "event record"))) return rc;
  if (pre) {
    eprop::InputArgs nx = ia;
    nx.x = x_next; nx.steps = steps_next; nx.Iin = P.Iin[ib ^ 1]; nx.nin = P.nin[ib ^ 1];
    if ((rc = check(ctx, hipStreamWaitEvent(ctx->in_stream, ctx->ev_pre, 0), "stream wait")) ||
        (rc = check(ctx, eprop::launch_input_drive(nx, ctx->in_stream), "input drive kernel")) ||
        (rc = check(ctx, hipEventRecord(ctx->ev_in[ib ^ 1], ctx->in_stream), "event record")))
      return rc;
    ctx->in_buf = ib ^ 1;
    ctx->in_ready = true;
  }

  // On the coefficient stream: the first layer's input filter and p bits,
  // then per layer the learning signal, the readout gradient and the block
  // coefficients of the eligibility recursion; the forward of the next block
  // (other slot) runs meanwhile.  Where an eligibility pass is long against
  // the block's forward (its trace round trip above a quarter of the forward
  // steps' cost), it waits for all of that: started earlier it would slow
  // the next forward, the longer path.  Where it is short, the eligibility
  // pass starts as early as it can: the input filter (it needs only x) is
  // queued ahead of the wait for the forward, and the readout gradient after
  // the coefficients, past the eligibility pass's wait.
  const SplitCost cost = split_cost(P);
  const bool early = ev && 4.0 * cost.round_trip_us < steps * cost.step_us;
  if (early) {
    if (ctx->slot_used[sl] &&
        (rc = check(ctx, hipStreamWaitEvent(sc, ctx->ev_done[sl], 0), "stream wait")))
      return rc;
    if ((rc = check(ctx, eprop::launch_input_filter(ia, sc), "input filter kernel"))) return rc;
  }
  if (ev && (rc = check(ctx, hipStreamWaitEvent(sc, ctx->ev_fwd[sl], 0), "stream wait"))) return rc;
  if (!early && (rc = check(ctx, eprop::launch_input_filter(ia, sc), "input filter kernel"))) return rc;
  const int rows = steps * P.Bp;
  const int kpad = (int)round_up(steps, 16);
  auto readout_gradient = [&](int l) {
    Layer& L = ctx->plan.layers[l];
    // dW_out += sum over (t, b) of delta (x) ztilde, then fp64 accumulation
    eprop::GemmArgs g;
    g.A = L.deltaK[sl]; g.Bm = L.ztK[sl]; g.C = L.Cpart;
    g.M = c.n_out; g.N = c.n_rec; g.K = rows; g.lda = P.ldk; g.ldb = P.ldn; g.ldc = c.n_rec;
    choose_splits(g.M, g.N, g.K, P.out_splits, &g.splits, &g.k_chunk);
    g.split_stride = (size_t)c.n_out * c.n_rec;
    int r = check(ctx, eprop::launch_gemm_tn(g, sc), "readout gradient GEMM");
    if (!r)
      r = check(ctx, eprop::launch_accumulate(L.Cpart, g.splits, g.split_stride, c.n_out, c.n_rec,
                                              L.accout, L.ldj, first, sc),
                "readout gradient accumulation");
    return r;
  };
  for (int l = 0; l < c.n_layers; ++l) {
    Layer& L = ctx->plan.layers[l];
    // learning signal L[(t,b)][j] = sum_k delta[(t,b)][k] W_out[k][j]
    eprop::GemmArgs gl;
    gl.A = L.deltaK[sl]; gl.Bm = L.Fb_src ? L.FbT : L.WoutT; gl.C = L.LK[sl];
    gl.M = rows; gl.N = c.n_rec; gl.K = P.ldk; gl.lda = P.ldk; gl.ldb = P.ldk; gl.ldc = L.ldv;
    gl.splits = 1; gl.k_chunk = P.ldk; gl.split_stride = 0;
    if ((rc = check(ctx, eprop::launch_gemm_nt(gl, sc), "learning-signal GEMM"))) return rc;
    if (!early && (rc = readout_gradient(l))) return rc;

    eprop::CoefArgs ca;
    ca.psiK = L.psiK[sl]; ca.LK = L.LK[sl]; ca.ldv = L.ldv; ca.Bp = P.Bp;
    ca.O = L.coefO[sl]; ca.ol = P.ol;
    ca.S = L.coefS[sl];
    ca.B = c.batch; ca.n_post = c.n_rec; ca.n_adaptive = c.n_adaptive;
    ca.steps = steps; ca.kpad = kpad; ca.ldc = P.ldc;
    ca.kappa = c.kappa; ca.rho = c.rho; ca.beta = c.beta; ca.alpha = c.alpha; ca.thr = c.thr;
    ca.reset_through = P.rt;
    ca.model = c.neuron_model;
    for (int m = 0; m < 2; ++m) {
      ca.gA[m][0] = (float)P.gen.A[m][0]; ca.gA[m][1] = (float)P.gen.A[m][1];
      ca.gb[m] = (float)P.gen.b[m]; ca.gr[m] = (float)P.gen.r[m]; ca.gc[m] = (float)P.gen.c[m];
    }
    if ((rc = check(ctx, eprop::launch_coef(ca, sc), "eligibility coefficient kernel"))) return rc;
  }
  if (ev && (rc = check(ctx, hipEventRecord(ctx->ev_coef[sl], sc), "event record"))) return rc;
  if (ev && (rc = check(ctx, hipStreamWaitEvent(s, ctx->ev_coef[sl], 0), "stream wait"))) return rc;
  for (int l = 0; early && l < c.n_layers; ++l)
    if ((rc = readout_gradient(l))) return rc;
  if (ev && (rc = check(ctx, hipEventRecord(ctx->ev_out[sl], sc), "event record"))) return rc;

  // On the caller's stream: the eligibility pass of every layer.
  for (int l = 0; l < c.n_layers; ++l) {
    const Layer& L = P.layers[l];
    eprop::TraceArgs ta;
    ta.ebar = L.ebar; ta.epsa = L.epsa; ta.epsv = L.epsv; ta.acc = L.acc; ta.acc_stride = L.acc_stride;
    ta.n_split = L.n_split; ta.pbits = L.pbits[sl];
    ta.zstart = L.zstart[sl];
    ta.O = L.coefO[sl]; ta.ol = P.ol; ta.reset_through = P.rt;
    ta.S = L.coefS[sl];
    ta.B = c.batch; ta.n_pre = L.n_pre; ta.n_pre_pad = L.n_pre_pad; ta.n_post = c.n_rec; ta.ldj = L.ldj;
    ta.n_adaptive = P.na2; ta.ldi = L.n_pre_pad;
    ta.n_jt = (c.n_rec + eprop::kTileJ - 1) / eprop::kTileJ;
    ta.n_jt_a = (P.na2 + eprop::kTileJ - 1) / eprop::kTileJ;
    ta.ldc = P.ldc; ta.kpad = kpad;
    ta.kappa_K = (float)std::pow((double)c.kappa, (double)steps);
    ta.first = first;
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
  // later work on the caller's stream (the next blocks, the gradient
  // read-out, an online update) and the reuse of this slot also follow the
  // readout gradient
  if (ev && (rc = check(ctx, hipStreamWaitEvent(s, ctx->ev_out[sl], 0), "stream wait"))) return rc;
  if (ev && (rc = check(ctx, hipEventRecord(ctx->ev_done[sl], s), "event record"))) return rc;
  ctx->slot_used[sl] = true;
  ctx->last_slot = sl;
  ctx->slot = (ctx->slot + 1) % P.slots;
  ctx->t += steps;
  ctx->last_steps = steps;
  return EPROP_OK;
}

bool usable(const eprop_ctx* ctx) { return ctx && ctx->alive; }

// Work queued on the caller's stream before this call (inputs, a reset, new
// weights) happens before the forward kernels of this call.
int join_forward_stream(eprop_ctx* ctx) {
  ctx->in_ready = false;   // an input drive is only computed ahead within a call
  if (ctx->single_stream) return EPROP_OK;
  int rc = check(ctx, hipEventRecord(ctx->ev_entry, ctx->stream), "event record");
  if (!rc) rc = check(ctx, hipStreamWaitEvent(ctx->fwd_stream, ctx->ev_entry, 0), "stream wait");
  return rc;
}

// Argument checks shared by eprop_init and eprop_sequence_static (errors
// reported through eprop_last_error(NULL)).
int check_init_args(const eprop_config* cfg, const void* d_workspace, size_t ws_bytes,
                    const float* const* d_weights, int slots = kSlots) {
  std::string why;
  if (!valid_config(cfg, &why)) return fail(nullptr, EPROP_EINVAL, why);
  if (!d_workspace || !d_weights) return fail(nullptr, EPROP_EINVAL, "workspace or weights is NULL");
  if (((uintptr_t)d_workspace) % 256 != 0)
    return fail(nullptr, EPROP_EINVAL, "workspace must be 256-byte aligned");
  for (int k = 0; k < 2 * cfg->n_layers; ++k)
    if (!d_weights[k]) return fail(nullptr, EPROP_EINVAL, "a weight pointer is NULL");
  Plan probe;
  make_plan(*cfg, nullptr, &probe, slots);
  if (!plan_fits(probe, &why)) return fail(nullptr, EPROP_EINVAL, why);
  if (ws_bytes < probe.bytes)
    return fail(nullptr, EPROP_ENOSPACE,
                "workspace too small: need " + std::to_string(probe.bytes) + " bytes");
  return EPROP_OK;
}

// Lays the context out in the workspace and queues the clear, the weight
// packing and the state reset.  With single_stream the context creates no
// streams or events: every kernel goes to the caller's stream in issue order.
int setup_ctx(eprop_ctx* ctx, const eprop_config* cfg, char* ws, size_t ws_bytes,
              const float* const* d_weights, hipStream_t stream, bool single_stream) {
  ctx->ws = ws;
  ctx->ws_bytes = ws_bytes;
  ctx->stream = stream;
  ctx->single_stream = single_stream;
  make_plan(*cfg, ctx->ws, &ctx->plan, single_stream ? 1 : kSlots);
  for (int l = 0; l < cfg->n_layers; ++l) {
    ctx->plan.layers[l].W_src = d_weights[2 * l];
    ctx->plan.layers[l].Wout_src = d_weights[2 * l + 1];
  }
  int rc = EPROP_OK;
  if (single_stream) {
    ctx->fwd_stream = ctx->coef_stream = stream;
  } else {
    rc = check(ctx, hipStreamCreateWithFlags(&ctx->fwd_stream, hipStreamNonBlocking), "stream create");
    if (!rc) rc = check(ctx, hipStreamCreateWithFlags(&ctx->coef_stream, hipStreamNonBlocking),
                        "stream create");
    if (!rc) rc = check(ctx, hipEventCreateWithFlags(&ctx->ev_entry, hipEventDisableTiming), "event create");
    if (!rc) rc = check(ctx, hipEventCreateWithFlags(&ctx->ev_update, hipEventDisableTiming), "event create");
    if (!rc) rc = check(ctx, hipStreamCreateWithFlags(&ctx->in_stream, hipStreamNonBlocking), "stream create");
    if (!rc) rc = check(ctx, hipEventCreateWithFlags(&ctx->ev_pre, hipEventDisableTiming), "event create");
    for (int k = 0; k < 2 && !rc; ++k)
      rc = check(ctx, hipEventCreateWithFlags(&ctx->ev_in[k], hipEventDisableTiming), "event create");
    for (int k = 0; k < kSlots && !rc; ++k) {
      rc = check(ctx, hipEventCreateWithFlags(&ctx->ev_fwd[k], hipEventDisableTiming), "event create");
      if (!rc) rc = check(ctx, hipEventCreateWithFlags(&ctx->ev_out[k], hipEventDisableTiming),
                          "event create");
      if (!rc) rc = check(ctx, hipEventCreateWithFlags(&ctx->ev_coef[k], hipEventDisableTiming),
                          "event create");
      if (!rc) rc = check(ctx, hipEventCreateWithFlags(&ctx->ev_done[k], hipEventDisableTiming),
                          "event create");
    }
  }
  // Padding of every buffer must read as zero; clear the whole layout once.
  if (!rc) rc = check(ctx, eprop::launch_zero(ctx->ws, ctx->plan.bytes, ctx->stream), "workspace clear");
  if (!rc) rc = pack_weights(ctx);
  if (!rc) rc = clear_state(ctx);
  if (!rc) ctx->alive = true;
  return rc;
}

// ---------------------------------------------------------------- static scratch
// Device memory of eprop_sequence_static: a file-scope array that every GPU
// the library runs on holds (its own copy) until the process ends.  Host code
// never passes the array's name to a kernel: its device address, per device,
// comes from hipGetSymbolAddress on the first call on that device.
constexpr size_t kScratchBytes = (size_t)EPROP_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The scratch array's address on the current device (set up once per device).
int scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(nullptr, EPROP_EDEVICE, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(nullptr, EPROP_EDEVICE, "device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(nullptr, EPROP_EDEVICE,
                  std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return EPROP_OK;
}

}  // namespace

extern "C" {

int eprop_neuron_coefficients(const eprop_config* cfg, int32_t cls, float* out) {
  std::string why;
  if (!valid_config(cfg, &why)) return fail(nullptr, EPROP_EINVAL, why);
  if (!out || (cls != 0 && cls != 1)) return fail(nullptr, EPROP_EINVAL, "out is NULL or cls not 0/1");
  NeuronCoef k;
  if (!derive_neuron(*cfg, cls, &k)) return fail(nullptr, EPROP_EINVAL, "neuron step is not linear in its state");
  const double v[10] = {k.A[0][0], k.A[0][1], k.A[1][0], k.A[1][1], k.b[0], k.b[1],
                        k.r[0], k.r[1], k.c[0], k.c[1]};
  for (int q = 0; q < 10; ++q) out[q] = (float)v[q];
  return EPROP_OK;
}

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
  int rc = check_init_args(cfg, d_workspace, ws_bytes, d_weights);
  if (rc) return rc;
  eprop_ctx* ctx = new eprop_ctx();
  rc = setup_ctx(ctx, cfg, (char*)d_workspace, ws_bytes, d_weights, (hipStream_t)hip_stream, false);
  if (rc) {
    g_last_error = ctx->err;
    eprop_destroy(ctx);
    return rc;
  }
  *out = ctx;
  return EPROP_OK;
}

int eprop_sequence_static(const eprop_config* cfg, const float* const* d_weights, const uint8_t* d_x,
                          int32_t T, const int32_t* d_labels, uint32_t* d_spikes,
                          float* const* d_grads, double* d_loss, void* hip_stream) {
  if (!d_x || !d_labels || !d_grads) return fail(nullptr, EPROP_EINVAL, "x, labels or grads is NULL");
  if (T < 1) return fail(nullptr, EPROP_EINVAL, "T must be >= 1");
  std::string why;
  if (!valid_config(cfg, &why)) return fail(nullptr, EPROP_EINVAL, why);
  for (int k = 0; k < 2 * cfg->n_layers; ++k)
    if (!d_grads[k]) return fail(nullptr, EPROP_EINVAL, "a gradient pointer is NULL");
  // the size check comes before any device call; everything runs on one
  // stream, so one set of per-block buffers is enough
  Plan probe;
  make_plan(*cfg, nullptr, &probe, 1);
  if (!plan_fits(probe, &why)) return fail(nullptr, EPROP_EINVAL, why);
  const size_t need = probe.bytes;
  if (need > kScratchBytes)
    return fail(nullptr, EPROP_ENOSPACE,
                "shape needs " + std::to_string(need) + " bytes of workspace; the static scratch holds " +
                    std::to_string(kScratchBytes));
  void* ws = nullptr;
  int rc = scratch_address(&ws);
  if (rc) return rc;
  rc = check_init_args(cfg, ws, kScratchBytes, d_weights, 1);
  if (rc) return rc;
  eprop_ctx ctx;   // host-side bookkeeping only, on this stack frame
  rc = setup_ctx(&ctx, cfg, (char*)ws, kScratchBytes, d_weights, (hipStream_t)hip_stream, true);
  if (!rc) rc = eprop_run_sequence(&ctx, d_x, T, d_labels, d_spikes);
  if (!rc) rc = eprop_get_grads(&ctx, d_grads, d_loss);
  if (rc) g_last_error = ctx.err;
  ctx.alive = false;
  return rc;
}

int eprop_step(eprop_ctx* ctx, const uint8_t* d_x_t, const int32_t* d_labels, uint32_t* d_spikes_t) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (!d_x_t || !d_labels) return fail(ctx, EPROP_EINVAL, "x or labels is NULL");
  int rc = join_forward_stream(ctx);
  if (rc) return rc;
  return do_block(ctx, d_x_t, 1, d_labels, d_spikes_t, nullptr, 0);
}

namespace {

// Blocks of up to Kmax steps that end where the weights change.  The steps
// up to the next change (or the end of the call), a segment, form one block
// when they are at most Kmax / 2, else blocks of equal length (within a
// step), at least two, so that the forward pass of the second block runs
// beside the eligibility pass of the first.  A segment of at most Kmax / 2
// (and at least 2 kMinHalf) steps is cut in two halves as well when the
// forward steps of a half cost more than one more trace round trip.  A segment longer than Kmax may
// instead start with a short block followed by k blocks of twice its length
// (k the smallest count that keeps those at most Kmax), when that adds one
// block to the equal split: the first eligibility pass then starts that many
// forward steps earlier, which pays when the steps saved cost more than the
// added trace round trip.
constexpr long long kMinHalf = 64;   // shortest half of a segment cut in two

struct Split {
  int32_t seg_end = 0;   // end of the current segment (call-local step)
  int blk = 0;           // length of its blocks after the first
};

int next_block(int32_t t, int32_t T, long long t_ctx, int32_t every, int mode,
               const SplitCost& cost, Split& sp) {
  if (t < sp.seg_end) return std::min(sp.blk, sp.seg_end - t);
  long long seg = T - t;
  if (every > 0) seg = std::min<long long>(seg, every - t_ctx % every);
  sp.seg_end = (int32_t)(t + seg);
  const long long K = kBlockSteps;
  long long first = seg, blk = seg;
  if (seg <= K / 2) {
    if (mode == EPROP_SPLIT_AUTO && seg >= 2 * kMinHalf && (double)(seg / 2) * cost.step_us > cost.round_trip_us)
      first = blk = (seg + 1) / 2;
  } else {
    const long long nb = std::max<long long>(2, (seg + K - 1) / K);
    first = blk = (seg + nb - 1) / nb;
    if (seg > K) {
      const long long k = (2 * seg - K + 2 * K - 1) / (2 * K);
      const long long short_first = (seg + 2 * k) / (2 * k + 1);
      if (mode == EPROP_SPLIT_AUTO && k == nb &&
          (double)(first - short_first) * cost.step_us > cost.round_trip_us) {
        first = short_first;
        blk = (seg - short_first + k - 1) / k;
      }
    }
  }
  sp.blk = (int)blk;
  return (int)first;
}

}  // namespace

int eprop_block_lengths(const eprop_config* cfg, int32_t T, int64_t t0, int32_t online_every,
                        int32_t mode, int32_t* lengths, int32_t max_blocks) {
  std::string why;
  if (!valid_config(cfg, &why)) return fail(nullptr, EPROP_EINVAL, why);
  if (T < 1 || t0 < 0 || online_every < 0 || max_blocks < 0 || (max_blocks > 0 && !lengths) ||
      (mode != EPROP_SPLIT_AUTO && mode != EPROP_SPLIT_EQUAL))
    return fail(nullptr, EPROP_EINVAL, "T must be >= 1, t0, online_every and max_blocks >= 0, "
                                       "lengths not NULL when max_blocks > 0, mode a split mode");
  Plan probe;
  make_plan(*cfg, nullptr, &probe);
  const SplitCost cost = split_cost(probe);
  Split sp;
  int32_t n = 0;
  for (int32_t t = 0; t < T; ++n) {
    const int steps = next_block(t, T, t0 + t, online_every, mode, cost, sp);
    if (n < max_blocks) lengths[n] = steps;
    t += steps;
  }
  return n;
}

int eprop_run_sequence(eprop_ctx* ctx, const uint8_t* d_x, int32_t T, const int32_t* d_labels,
                       uint32_t* d_spikes) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (!d_x || !d_labels) return fail(ctx, EPROP_EINVAL, "x or labels is NULL");
  if (T < 1) return fail(ctx, EPROP_EINVAL, "T must be >= 1");
  const eprop_config& c = ctx->plan.cfg;
  const size_t x_step = (size_t)c.batch * c.n_in;
  const size_t s_step = (size_t)c.n_layers * c.batch * ((c.n_rec + 31) / 32);
  int rc0 = join_forward_stream(ctx);
  if (rc0) return rc0;
  const SplitCost cost = split_cost(ctx->plan);
  Split sp;
  for (int32_t t = 0; t < T;) {
    const int steps = next_block(t, T, ctx->t, ctx->online_every, ctx->split_mode, cost, sp);
    const int32_t tn = t + steps;
    Split sp_next = sp;
    const int steps_next =
        tn < T ? next_block(tn, T, ctx->t + steps, ctx->online_every, ctx->split_mode, cost, sp_next) : 0;
    int rc = do_block(ctx, d_x + t * x_step, steps, d_labels,
                      d_spikes ? d_spikes + t * s_step : nullptr,
                      steps_next > 0 ? d_x + tn * x_step : nullptr, steps_next);
    if (rc) return rc;
    t = tn;
  }
  return EPROP_OK;
}

int eprop_get_grads(eprop_ctx* ctx, float* const* d_grads, double* d_loss) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (!d_grads) return fail(ctx, EPROP_EINVAL, "grads is NULL");
  const eprop_config& c = ctx->plan.cfg;
  for (int k = 0; k < 2 * c.n_layers; ++k)
    if (!d_grads[k]) return fail(ctx, EPROP_EINVAL, "a gradient pointer is NULL");
  eprop::ReadoutArgs ro{};
  ro.n_layers = c.n_layers;
  for (int l = 0; l < c.n_layers; ++l) {
    Layer& L = ctx->plan.layers[l];
    eprop::GradsArgs& g = ro.g[l];
    g.acc = L.acc; g.ldj = L.ldj; g.n_split = L.n_split; g.acc_stride = L.acc_stride;
    g.dW = d_grads[2 * l]; g.n_pre = L.n_pre; g.n_post = c.n_rec;
    g.n_inl = L.n_inl; g.recurrent = c.recurrent;
    g.accout = L.accout; g.ld_acc = L.ldj; g.dWout = d_grads[2 * l + 1]; g.K = c.n_out;
    g.valid = ctx->t > 0;
  }
  if (d_loss) {
    const Layer& L0 = ctx->plan.layers[0];
    ro.lossacc = L0.lossacc;
    ro.B = c.batch;
    ro.layer_stride = c.n_layers > 1 ? (size_t)(ctx->plan.layers[1].lossacc - L0.lossacc) : 0;
    ro.loss = d_loss;
  }
  int rc = check(ctx, eprop::launch_readout(ro, ctx->stream), "gradient read-out");
  if (rc) return rc;
  return EPROP_OK;
}

int eprop_reset(eprop_ctx* ctx) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  int rc = pack_weights(ctx);
  if (!rc) rc = pack_feedback(ctx);
  if (!rc) rc = clear_state(ctx);
  return rc;
}

int eprop_set_feedback(eprop_ctx* ctx, const float* const* d_feedback) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  for (int l = 0; l < ctx->plan.cfg.n_layers; ++l)
    ctx->plan.layers[l].Fb_src = d_feedback ? d_feedback[l] : nullptr;
  // Queued after the work already enqueued: the blocks of earlier calls
  // (whose learning-signal GEMMs read the old matrices) run before the
  // repacking, because the coefficient stream is joined to the caller's
  // stream by every block's eligibility pass.
  return pack_feedback(ctx);
}

int eprop_set_online(eprop_ctx* ctx, float lr, int32_t every) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (every < 0 || !std::isfinite(lr)) return fail(ctx, EPROP_EINVAL, "every must be >= 0 and lr finite");
  ctx->online_lr = lr;
  ctx->online_every = every;
  return EPROP_OK;
}

int eprop_set_block_split(eprop_ctx* ctx, int32_t mode) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (mode != EPROP_SPLIT_AUTO && mode != EPROP_SPLIT_EQUAL)
    return fail(ctx, EPROP_EINVAL, "mode must be EPROP_SPLIT_AUTO or EPROP_SPLIT_EQUAL");
  ctx->split_mode = mode;
  return EPROP_OK;
}

int eprop_get_weights(eprop_ctx* ctx, float* const* d_weights) {
  if (!usable(ctx)) return fail(ctx, EPROP_ESTATE, "context not initialised");
  if (!d_weights) return fail(ctx, EPROP_EINVAL, "weights is NULL");
  const eprop_config& c = ctx->plan.cfg;
  for (int k = 0; k < 2 * c.n_layers; ++k)
    if (!d_weights[k]) return fail(ctx, EPROP_EINVAL, "a weight pointer is NULL");
  for (int l = 0; l < c.n_layers; ++l) {
    const Layer& L = ctx->plan.layers[l];
    int rc = check(ctx, eprop::launch_unpack_weights(L.Wt, L.ldw, L.WoutT, ctx->plan.ldk, c.n_rec,
                                                     L.n_pre, c.n_out, d_weights[2 * l],
                                                     d_weights[2 * l + 1], ctx->stream),
                   "weight read-out");
    if (rc) return rc;
  }
  return EPROP_OK;
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
  for (hipStream_t st : {ctx->fwd_stream, ctx->coef_stream, ctx->in_stream}) {
    if (!st || ctx->single_stream) continue;   // the caller's stream is not ours
    (void)hipStreamSynchronize(st);
    (void)hipStreamDestroy(st);
  }
  if (ctx->ev_entry) (void)hipEventDestroy(ctx->ev_entry);
  if (ctx->ev_update) (void)hipEventDestroy(ctx->ev_update);
  for (hipEvent_t e : {ctx->ev_pre, ctx->ev_in[0], ctx->ev_in[1]})
    if (e) (void)hipEventDestroy(e);
  for (int k = 0; k < kSlots; ++k)
    for (hipEvent_t e : {ctx->ev_fwd[k], ctx->ev_coef[k], ctx->ev_out[k], ctx->ev_done[k]})
      if (e) (void)hipEventDestroy(e);
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
  // psiK and LK rows are t*Bp + b: the last step's rows start at (last_steps-1)*Bp
  const int64_t tl = (int64_t)(ctx->last_steps - 1) * ctx->plan.Bp;
  switch (which) {
    case 0: *d_ptr = L.v; *cols = c.n_rec; *ld = c.n_rec; break;
    case 1: *d_ptr = L.a; *cols = c.n_rec; *ld = c.n_rec; break;
    case 2: *d_ptr = L.psiK[ctx->last_slot] + tl * L.ldv; *cols = c.n_rec; *ld = L.ldv; break;
    case 3: *d_ptr = L.LK[ctx->last_slot] + tl * L.ldv; *cols = c.n_rec; *ld = L.ldv; break;
    case 4: *d_ptr = L.y; *cols = c.n_out; *ld = c.n_out; break;
    case 5: *d_ptr = reinterpret_cast<const float*>(ctx->plan.w16ok); *cols = 2; *ld = 2; break;
    default: return fail(ctx, EPROP_EINVAL, "unknown buffer");
  }
  return EPROP_OK;
}

}  // extern "C"
