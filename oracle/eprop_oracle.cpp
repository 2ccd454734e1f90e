// TEST INFRASTRUCTURE ONLY -- the CPU oracle of the online e-prop step.
//
// A plain, slow, single-threaded implementation of what the hot path computes,
// written from the paper (arxiv 2501.11407).  Only the test suite, the smoke
// check and the benchmark's CPU-baseline leg may load this library.  It shares
// no code, header or constant with the HIP library; the two meet only in the
// seeded inputs.
//
// What it computes, per batch element b, per timestep t, per layer:
//   * the LIF neuron of Eq. (8a,b) with an adaptive threshold (ALIF) on the
//     first n_adaptive neurons, reset by subtraction, input x^t entering v^t
//     in the same step and the recurrent spikes z^{t-1} entering one step
//     later;
//   * the non-spiking leaky readout with a softmax cross-entropy loss at every
//     step, the loss being the sum over steps of Eq. (2);
//   * the gradient of Eq. (3) accumulated forward in time with the RTRL
//     recursion of Eq. (5), G_t = H_t G_{t-1} + F_t, in which H_t keeps only
//     the neuron-on-itself part H_{I,t} (Sec. III-B: the recurrent spikes are
//     gradient-stopped).  H_{I,t} is then diagonal over neurons, with a 2x2
//     block [[alpha, 0], [psi, rho - beta*psi]] per adaptive neuron (the
//     block-diagonal case of the footnote in Sec. III-C), and F_t = dh_t/dW_ji
//     is the presynaptic value p_i^t, so the matrix product of Eq. (5) becomes
//     an element-wise update of per-synapse eligibility vectors (Sec. III-B).
//     The product dL/dh_t G_t is the eligibility trace of Sec. III-B.
//
// Readings of points the paper leaves open (each is also listed in the design
// notes of the repository):
//   * the reset path (own spike -> own membrane) is gradient-stopped like the
//     recurrent spikes; the spike -> adaptation path is kept;
//   * ALIF: A = thr + beta*a, a^t = rho*a^{t-1} + z^{t-1};
//   * surrogate (footnote in Sec. III-C): psi = (gamma/thr)*max(0, 1-|v-A|/thr);
//   * spike iff v - A > 0 strictly; reset subtracts `reset` (= thr);
//   * readout y^t = kappa*y^{t-1} + W_out z^t, no bias; learning signal
//     L = W_out^T (softmax(y) - onehot(label)); the kappa filter of the readout
//     moves onto the trace (ebar), which makes the forward sum exact;
//   * optional fixed feedback: L = B^T (softmax(y) - onehot(label)) with a
//     matrix B of W_out's shape in place of W_out (random feedback weights,
//     the readout approximation that the source of Sec. III-B names and sets
//     aside); only the learning signal changes;
//   * two-layer stacks: layer 2 reads layer-1 spikes of the same step,
//     gradient-stopped, and has its own readout and loss;
//   * the recurrent-weight diagonal (no self-connections) gets gradient 0;
//   * optionally (reset_through) the reset path is kept in the gradient: the
//     own spike z^{t-1} = H(v - A) then carries dv^t/dv^{t-1} = alpha -
//     reset*psi^{t-1} and dv^t/da^{t-1} = reset*beta*psi^{t-1}, so the
//     membrane component of G_t is a per-synapse eps^v (no longer the
//     presynaptic filter zbar): one of the neuron-model variants the generic
//     method of Sec. III-C covers.
//   * optionally (model = 1) a two-compartment neuron instead: a dendrite d
//     that receives the synaptic drive and the neuron's own last spike (a
//     backpropagating spike of strength q, kept in the gradient), and a soma
//     s driven by the dendrite's previous value through a coupling g and
//     reset by subtraction:
//       d^t = alpha_d d^{t-1} + I^t + q z^{t-1}
//       s^t = alpha s^{t-1} + g d^{t-1} - reset z^{t-1}
//       z^t = H(s^t - thr),  psi^t = (gamma/thr) max(0, 1 - |s^t - thr|/thr)
//     Its neuron-on-itself Jacobian is a full 2x2 block per neuron,
//     H_I^t = [[alpha - reset*psi^{t-1} (reset kept only), g],
//              [q psi^{t-1}, alpha_d]]  over (s, d),
//     and F_t = dh^t/dW_ji = (0, p_i^t): the block-diagonal case of the
//     footnote in Sec. III-C with a state-dependent off-diagonal, so both
//     components of the eligibility vector are per-synapse state.
//
// Precision: the neuron state (v, a, A, v-A) and the spike decision are
// computed in the type R chosen by `fwd_fp32` (fp32 like the paper's runs,
// or fp64 for the checks against reverse-mode autograd), one rounding per
// written operation and no contraction (build with -ffp-contract=off).
// Everything on the gradient path is fp64.

#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <vector>

extern "C" {

typedef struct {
  int32_t n_layers;    // 1 or 2
  int32_t batch;       // B
  int32_t n_in;        // inputs of layer 0
  int32_t n_rec;       // neurons per layer
  int32_t n_out;       // readout classes K
  int32_t recurrent;   // 0: presynaptic vector is the layer input alone
  int32_t n_adaptive;  // neurons j < n_adaptive are ALIF
  double alpha, rho, kappa, thr, beta, gamma;
  double reset;        // amount subtracted from v after a spike
  int32_t fwd_fp32;    // 1: neuron state and spike decision in fp32, 0: fp64
  int32_t smooth;      // 1: z = S(v-A) with S' = psi (finite-difference checks)
  int32_t reset_through;  // 1: the reset path (own spike -> own membrane) is kept
  int32_t model;       // 0: LIF/ALIF, 1: two-compartment neuron (soma s, dendrite d)
  double alpha_d;      // model 1: dendritic decay
  double coupling;     // model 1: dendrite -> soma coupling g
  double bap;          // model 1: own spike -> dendrite (backpropagating spike) q
} oracle_config;

// Optional per-step records; each pointer may be NULL.
// v, a, psi, L, z: [T][n_layers][B][n_rec]; y: [T][n_layers][B][n_out].
typedef struct {
  double* v;
  double* a;
  double* psi;
  double* L;
  double* z;
  double* y;
} oracle_record;

}  // extern "C"

namespace {

struct Synapse {  // one sampled synapse: W^{(layer)}[j][i]
  int32_t layer, j, i;
};

// Integral of the triangular surrogate: S' = psi.  Used only in smooth mode.
double smooth_spike(double x, double thr, double gamma) {
  double u = x / thr;
  if (u <= -1.0) return 0.0;
  if (u <= 0.0) return gamma * 0.5 * (1.0 + u) * (1.0 + u);
  if (u < 1.0) return gamma * (0.5 + u - 0.5 * u * u);
  return gamma;
}

template <typename R>
struct LayerState {
  int n_in_l = 0, n_pre = 0;
  std::vector<R> v, a;             // membrane potential, threshold adaptation
  std::vector<double> z, z_prev;   // spikes at t and t-1
  std::vector<double> p;           // presynaptic vector [x^t ; z^{t-1}]
  std::vector<double> zbar;        // alpha-filtered p: the eps^v component of G_t
  std::vector<double> psi;         // pseudo-derivative dz/d(v-A)
  std::vector<double> y, ztil;     // readout potential, kappa-filtered spikes
  std::vector<double> delta, L;    // dCE/dy, learning signal W_out^T delta
  std::vector<double> ebar, epsa;  // eligibility: kappa-filtered trace, eps^a
  std::vector<double> epsv;        // per-synapse eps^v (reset_through; without the next input)
  // two-compartment neuron: per-synapse eligibility vector (eps_s, eps_d) of
  // the last step, and the pseudo-derivative of the last step per neuron
  std::vector<double> eps_s, eps_d, psi_prev;
};

// The state of one batch element: neuron state, filters and traces of every
// layer (and the traces of the sampled synapses).
template <typename R>
struct Seq {
  std::vector<LayerState<R>> st;
  std::vector<double> ebar_s, epsa_s, epsv_s;
};

template <typename R>
void seq_alloc(const oracle_config& c, bool all, int n_sample, Seq<R>& q) {
  const int NL = c.n_layers, N = c.n_rec, K = c.n_out, NA = c.n_adaptive;
  std::vector<LayerState<R>>& st = q.st;
  std::vector<double>& ebar_s = q.ebar_s;
  std::vector<double>& epsa_s = q.epsa_s;
  std::vector<double>& epsv_s = q.epsv_s;
  st.assign(NL, LayerState<R>());
  for (int l = 0; l < NL; ++l) {
    LayerState<R>& s = st[l];
    s.n_in_l = (l == 0) ? c.n_in : N;
    s.n_pre = s.n_in_l + (c.recurrent ? N : 0);
    s.v.assign(N, 0);
    s.a.assign(N, 0);
    s.z.assign(N, 0.0);
    s.z_prev.assign(N, 0.0);
    s.p.assign(s.n_pre, 0.0);
    s.zbar.assign(s.n_pre, 0.0);
    s.psi.assign(N, 0.0);
    s.y.assign(K, 0.0);
    s.ztil.assign(N, 0.0);
    s.delta.assign(K, 0.0);
    s.L.assign(N, 0.0);
    if (all) {
      s.ebar.assign((size_t)N * s.n_pre, 0.0);
      s.epsa.assign((size_t)NA * s.n_pre, 0.0);
      if (c.reset_through) s.epsv.assign((size_t)N * s.n_pre, 0.0);
      if (c.model == 1) {
        s.eps_s.assign((size_t)N * s.n_pre, 0.0);
        s.eps_d.assign((size_t)N * s.n_pre, 0.0);
      }
    }
    s.psi_prev.assign(N, 0.0);
  }
  if (!all) {
    ebar_s.assign(n_sample, 0.0);
    epsa_s.assign(n_sample, 0.0);
    epsv_s.assign(n_sample, 0.0);
  }
}


// A new sequence: every state, trace and filter starts at zero (G_0 = 0).
template <typename R>
void seq_zero(const oracle_config& c, Seq<R>& q) {
  const int NL = c.n_layers;
  std::vector<LayerState<R>>& st = q.st;
  for (int l = 0; l < NL; ++l) {
    LayerState<R>& s = st[l];
    std::fill(s.v.begin(), s.v.end(), R(0));
    std::fill(s.a.begin(), s.a.end(), R(0));
    std::fill(s.z.begin(), s.z.end(), 0.0);
    std::fill(s.z_prev.begin(), s.z_prev.end(), 0.0);
    std::fill(s.zbar.begin(), s.zbar.end(), 0.0);
    std::fill(s.y.begin(), s.y.end(), 0.0);
    std::fill(s.ztil.begin(), s.ztil.end(), 0.0);
    std::fill(s.ebar.begin(), s.ebar.end(), 0.0);
    std::fill(s.epsa.begin(), s.epsa.end(), 0.0);
    std::fill(s.epsv.begin(), s.epsv.end(), 0.0);
    std::fill(s.eps_s.begin(), s.eps_s.end(), 0.0);
    std::fill(s.eps_d.begin(), s.eps_d.end(), 0.0);
    std::fill(s.psi_prev.begin(), s.psi_prev.end(), 0.0);
  }
  std::fill(q.ebar_s.begin(), q.ebar_s.end(), 0.0);
  std::fill(q.epsa_s.begin(), q.epsa_s.end(), 0.0);
  std::fill(q.epsv_s.begin(), q.epsv_s.end(), 0.0);
}

// Steps t_lo .. t_hi-1 of batch element b from the state q, adding the
// gradient into dW, dWout and the loss into loss_sum (in step order).
template <typename R>
void steps(const oracle_config& c, const float* const* W, const float* const* Wout,
           const float* const* Fb, const uint8_t* x, int b, int label, int t_lo, int t_hi,
           const Synapse* sample, int n_sample, uint32_t* spikes, double* const* dW,
           double* const* dWout, double& loss_sum, const oracle_record* rec, Seq<R>& q,
           std::vector<int>& active) {
  const int NL = c.n_layers, B = c.batch, N = c.n_rec, K = c.n_out, NA = c.n_adaptive;
  const int W32 = (N + 31) / 32;
  const bool all = n_sample < 0;
  std::vector<LayerState<R>>& st = q.st;
  std::vector<double>& ebar_s = q.ebar_s;
  std::vector<double>& epsa_s = q.epsa_s;
  std::vector<double>& epsv_s = q.epsv_s;
  for (int t = t_lo; t < t_hi; ++t) {
    for (int l = 0; l < NL; ++l) {
      LayerState<R>& s = st[l];
      const float* Wl = W[l];
      const float* Wo = Wout[l];
      const float* Fo = (Fb && Fb[l]) ? Fb[l] : Wo;   // feedback matrix of the learning signal

      // Presynaptic vector p^t = [input^t ; z^{t-1}] and its alpha filter:
      // the eps^v component of G_t, since dv/dv = alpha and dv/dW_ji = p_i.
      for (int i = 0; i < s.n_in_l; ++i)
        s.p[i] = (l == 0) ? (x[((size_t)t * B + b) * c.n_in + i] ? 1.0 : 0.0) : st[l - 1].z[i];
      if (c.recurrent)
        for (int j = 0; j < N; ++j) s.p[s.n_in_l + j] = s.z_prev[j];
      for (int i = 0; i < s.n_pre; ++i) s.zbar[i] = c.alpha * s.zbar[i] + s.p[i];

      // Drive I_j = sum_i W_ji p_i.  Terms with p_i = 0 add nothing, so only
      // the nonzero entries are visited, in ascending i.
      active.clear();
      for (int i = 0; i < s.n_pre; ++i)
        if (s.p[i] != 0.0) active.push_back(i);

      // Neuron step, Eq. (8) with reset and adaptation, in precision R.
      const R alpha = (R)c.alpha, rho = (R)c.rho, thr = (R)c.thr, reset = (R)c.reset;
      for (int j = 0; j < N; ++j) {
        R I = 0;
        for (int i : active) I = I + (R)Wl[(size_t)j * s.n_pre + i] * (R)s.p[i];
        const R zp = (R)s.z_prev[j];
        R xj;
        if (c.model == 1) {
          // two-compartment neuron: v holds the soma s, a the dendrite d
          R d = (R)c.alpha_d * s.a[j];
          d = d + I;
          d = d + (R)c.bap * zp;
          R sm = alpha * s.v[j];
          sm = sm + (R)c.coupling * s.a[j];
          sm = sm - reset * zp;
          xj = sm - thr;
          s.v[j] = sm;
          s.a[j] = d;
        } else {
        R v = alpha * s.v[j];
        v = v + I;
        v = v - reset * zp;
        R a = rho * s.a[j];
        a = a + zp;
        const R bj = (j < NA) ? (R)c.beta : R(0);
        R A = bj * a;
        A = thr + A;
        xj = v - A;
        s.v[j] = v;
        s.a[j] = a;
        }
        const double xd = (double)xj;
        s.z[j] = c.smooth ? smooth_spike(xd, c.thr, c.gamma) : (xj > R(0) ? 1.0 : 0.0);
        const double u = 1.0 - std::fabs(xd) / c.thr;
        s.psi[j] = (c.gamma / c.thr) * (u > 0.0 ? u : 0.0);
      }

      // Leaky readout, softmax cross-entropy, learning signal, readout gradient.
      for (int k = 0; k < K; ++k) {
        double Y = 0.0;
        for (int j = 0; j < N; ++j)
          if (s.z[j] != 0.0) Y += (double)Wo[(size_t)k * N + j] * s.z[j];
        s.y[k] = c.kappa * s.y[k] + Y;
      }
      double m = s.y[0];
      for (int k = 1; k < K; ++k) m = s.y[k] > m ? s.y[k] : m;
      double se = 0.0;
      for (int k = 0; k < K; ++k) se += std::exp(s.y[k] - m);
      for (int k = 0; k < K; ++k)
        s.delta[k] = std::exp(s.y[k] - m) / se - (k == label ? 1.0 : 0.0);
      loss_sum += std::log(se) - (s.y[label] - m);
      for (int j = 0; j < N; ++j) {
        double Lj = 0.0;
        for (int k = 0; k < K; ++k) Lj += (double)Fo[(size_t)k * N + j] * s.delta[k];
        s.L[j] = Lj;
        s.ztil[j] = c.kappa * s.ztil[j] + s.z[j];
      }
      for (int k = 0; k < K; ++k)
        for (int j = 0; j < N; ++j) dWout[l][(size_t)k * N + j] += s.delta[k] * s.ztil[j];

      // Eligibility vectors and gradient accumulation (Eq. 5 with diagonal H,
      // then Eq. 3).  For synapse (j,i):
      //   e      = psi_j (zbar_i - beta_j epsa_ji)     dz_j^t/dW_ji
      //   ebar   = kappa ebar + e                      readout filter moved onto e
      //   dW_ji += L_j ebar
      //   epsa   = psi_j zbar_i + (rho - beta_j psi_j) epsa   (eps^a at t+1)
      // With the reset path kept, zbar_i is replaced by the per-synapse
      //   epsv   = epsv + p_i                              (eps^v at t)
      // and after the step
      //   epsv   = (alpha - reset psi_j) epsv + reset beta_j psi_j epsa
      //   epsa   = psi_j epsv + (rho - beta_j psi_j) epsa  (both with the values at t).
      if (c.model == 1) {
        // Eq. (5) with the 2x2 block H_I^t of each neuron (psi of the last
        // step in its second row, and in its first with the reset kept) and
        // F_t = (0, p_i): eps^t = H_I^t eps^{t-1} + F_t, then
        // e = dz^t/dW_ji = psi^t eps_s^t (z depends on the soma only).
        for (int q = 0; q < (all ? N * s.n_pre : n_sample); ++q) {
          int j, i;
          if (all) {
            j = q / s.n_pre;
            i = q - j * s.n_pre;
          } else {
            if (sample[q].layer != l) continue;
            j = sample[q].j;
            i = sample[q].i;
          }
          const double pp = s.psi_prev[j];
          const double h11 = c.alpha - (c.reset_through ? c.reset * pp : 0.0);
          const double h12 = c.coupling, h21 = c.bap * pp, h22 = c.alpha_d;
          const size_t ji = (size_t)j * s.n_pre + i;
          double& es = all ? s.eps_s[ji] : epsv_s[q];
          double& ed = all ? s.eps_d[ji] : epsa_s[q];
          double& eb = all ? s.ebar[ji] : ebar_s[q];
          const double es_new = h11 * es + h12 * ed;
          const double ed_new = h21 * es + h22 * ed + s.p[i];
          es = es_new;
          ed = ed_new;
          const double e = s.psi[j] * es;
          eb = c.kappa * eb + e;
          (all ? dW[l][ji] : dW[0][q]) += s.L[j] * eb;
        }
        for (int j = 0; j < N; ++j) s.psi_prev[j] = s.psi[j];
      } else if (c.reset_through) {
        for (int q = 0; q < (all ? N * s.n_pre : n_sample); ++q) {
          int j, i;
          if (all) {
            j = q / s.n_pre;
            i = q - j * s.n_pre;
          } else {
            if (sample[q].layer != l) continue;
            j = sample[q].j;
            i = sample[q].i;
          }
          const bool adaptive = j < NA;
          const double bj = adaptive ? c.beta : 0.0;
          const double pj = s.psi[j];
          const size_t ji = (size_t)j * s.n_pre + i;
          double& ev = all ? s.epsv[ji] : epsv_s[q];
          double& eb = all ? s.ebar[ji] : ebar_s[q];
          double* eap = adaptive ? (all ? &s.epsa[ji] : &epsa_s[q]) : nullptr;
          const double ea = eap ? *eap : 0.0;
          const double V = ev + s.p[i];
          const double e = pj * (V - bj * ea);
          eb = c.kappa * eb + e;
          (all ? dW[l][ji] : dW[0][q]) += s.L[j] * eb;
          ev = (c.alpha - c.reset * pj) * V + c.reset * bj * pj * ea;
          if (eap) *eap = pj * V + (c.rho - bj * pj) * ea;
        }
      } else if (all) {
        for (int j = 0; j < N; ++j) {
          const bool adaptive = j < NA;
          const double bj = adaptive ? c.beta : 0.0;
          const double pj = s.psi[j], Lj = s.L[j];
          for (int i = 0; i < s.n_pre; ++i) {
            const size_t ji = (size_t)j * s.n_pre + i;
            const double ea = adaptive ? s.epsa[ji] : 0.0;
            const double e = pj * (s.zbar[i] - bj * ea);
            s.ebar[ji] = c.kappa * s.ebar[ji] + e;
            dW[l][ji] += Lj * s.ebar[ji];
            if (adaptive) s.epsa[ji] = pj * s.zbar[i] + (c.rho - bj * pj) * ea;
          }
        }
      } else {
        for (int q = 0; q < n_sample; ++q) {
          if (sample[q].layer != l) continue;
          const int j = sample[q].j, i = sample[q].i;
          const bool adaptive = j < NA;
          const double bj = adaptive ? c.beta : 0.0;
          const double pj = s.psi[j];
          const double ea = adaptive ? epsa_s[q] : 0.0;
          const double e = pj * (s.zbar[i] - bj * ea);
          ebar_s[q] = c.kappa * ebar_s[q] + e;
          dW[0][q] += s.L[j] * ebar_s[q];
          if (adaptive) epsa_s[q] = pj * s.zbar[i] + (c.rho - bj * pj) * ea;
        }
      }

      if (spikes) {
        uint32_t* row = spikes + (((size_t)t * NL + l) * B + b) * W32;
        for (int w = 0; w < W32; ++w) row[w] = 0;
        for (int j = 0; j < N; ++j)
          if (s.z[j] > 0.0) row[j / 32] |= 1u << (j % 32);
      }
      if (rec) {
        const size_t o = (((size_t)t * NL + l) * B + b) * N;
        for (int j = 0; j < N; ++j) {
          if (rec->v) rec->v[o + j] = (double)s.v[j];
          if (rec->a) rec->a[o + j] = (double)s.a[j];
          if (rec->psi) rec->psi[o + j] = s.psi[j];
          if (rec->L) rec->L[o + j] = s.L[j];
          if (rec->z) rec->z[o + j] = s.z[j];
        }
        if (rec->y)
          for (int k = 0; k < K; ++k)
            rec->y[(((size_t)t * NL + l) * B + b) * K + k] = s.y[k];
      }
    }
    for (int l = 0; l < NL; ++l) st[l].z_prev = st[l].z;
  }
}

// No self-connections: the recurrent diagonal is not a parameter.
void zero_diagonal(const oracle_config& c, bool all, const Synapse* sample, int n_sample,
                   double* const* dW) {
  const int NL = c.n_layers, N = c.n_rec;
  if (all && c.recurrent)
    for (int l = 0; l < NL; ++l) {
      const int n_in_l = (l == 0) ? c.n_in : N;
      const int n_pre = n_in_l + N;
      for (int j = 0; j < N; ++j) dW[l][(size_t)j * n_pre + n_in_l + j] = 0.0;
    }
  if (!all)
    for (int q = 0; q < n_sample; ++q) {
      const int n_in_l = (sample[q].layer == 0) ? c.n_in : N;
      if (c.recurrent && sample[q].i == n_in_l + sample[q].j) dW[0][q] = 0.0;
    }
}

template <typename R>
int run(const oracle_config& c, const float* const* W, const float* const* Wout,
        const float* const* Fb, const uint8_t* x, int T, const int32_t* labels, int b_lo, int b_hi,
        const Synapse* sample, int n_sample, uint32_t* spikes, double* const* dW,
        double* const* dWout, double* loss, const oracle_record* rec) {
  const bool all = n_sample < 0;
  double loss_sum = 0.0;
  Seq<R> q;
  seq_alloc(c, all, n_sample, q);
  std::vector<int> active;
  for (int b = b_lo; b < b_hi; ++b) {
    seq_zero(c, q);
    steps(c, W, Wout, Fb, x, b, labels[b], 0, T, sample, n_sample, spikes, dW, dWout, loss_sum, rec,
          q, active);
  }
  zero_diagonal(c, all, sample, n_sample, dW);
  *loss += loss_sum;
  return 0;
}

// Online weight application: the gradient is available at every step
// (Sec. III-A), so the weights may change within the sequence.  Every `every`
// steps from the start, once every batch element has run them, the drive and
// readout weights in use become W0 - lr * G rounded to the nearest multiple
// of 2^-14 (ties to even), G being the gradient accumulated so far over all
// elements and steps; the recurrent diagonal keeps its W0 value.  All batch
// elements advance together, block by block, so each keeps its own state.
// Fixed feedback matrices (Fb, as in steps()) are not weights of the network:
// they keep their values while W and W_out change.
float on_grid(double v) { return (float)(std::nearbyint(v * 16384.0) / 16384.0); }

template <typename R>
int run_online(const oracle_config& c, const float* const* W0, const float* const* Wout0,
               const float* const* Fb, const uint8_t* x, int T, const int32_t* labels, double lr,
               int every,
               uint32_t* spikes, double* const* dW, double* const* dWout, double* loss,
               float* const* Wcur, float* const* Woutcur) {
  const int NL = c.n_layers, B = c.batch, N = c.n_rec, K = c.n_out;
  for (int l = 0; l < NL; ++l) {
    const size_t n_pre = (size_t)((l == 0) ? c.n_in : N) + (c.recurrent ? N : 0);
    std::memcpy(Wcur[l], W0[l], sizeof(float) * N * n_pre);
    std::memcpy(Woutcur[l], Wout0[l], sizeof(float) * (size_t)K * N);
  }
  std::vector<Seq<R>> qs(B);
  for (Seq<R>& q : qs) {
    seq_alloc(c, true, -1, q);
    seq_zero(c, q);
  }
  std::vector<double> loss_b(B, 0.0);
  std::vector<int> active;
  for (int t0 = 0; t0 < T; t0 += every) {
    const int t1 = t0 + every < T ? t0 + every : T;
    for (int b = 0; b < B; ++b)
      steps(c, Wcur, Woutcur, Fb, x, b, labels[b], t0, t1, nullptr, -1, spikes, dW, dWout,
            loss_b[b], nullptr, qs[b], active);
    if (t1 == T) break;
    for (int l = 0; l < NL; ++l) {
      const int n_in_l = (l == 0) ? c.n_in : N;
      const int n_pre = n_in_l + (c.recurrent ? N : 0);
      for (int j = 0; j < N; ++j)
        for (int i = 0; i < n_pre; ++i) {
          if (c.recurrent && i == n_in_l + j) continue;
          const size_t ji = (size_t)j * n_pre + i;
          Wcur[l][ji] = on_grid((double)W0[l][ji] - lr * dW[l][ji]);
        }
      for (size_t kj = 0; kj < (size_t)K * N; ++kj)
        Woutcur[l][kj] = on_grid((double)Wout0[l][kj] - lr * dWout[l][kj]);
    }
  }
  zero_diagonal(c, true, nullptr, -1, dW);
  double total = 0.0;
  for (int b = 0; b < B; ++b) total += loss_b[b];
  *loss += total;
  return 0;
}

bool valid(const oracle_config* c) {
  return c && (c->n_layers == 1 || c->n_layers == 2) && c->batch > 0 && c->n_in > 0 &&
         c->n_rec > 0 && c->n_out > 0 && c->n_adaptive >= 0 && c->n_adaptive <= c->n_rec &&
         c->thr > 0.0 && (c->model == 0 || (c->model == 1 && c->n_adaptive == 0));
}

}  // namespace

extern "C" {

// Bytes of state the oracle allocates for one run (one batch element at a
// time).  T does not enter: e-prop state is independent of sequence length.
size_t oracle_state_bytes(const oracle_config* c, int32_t n_sample) {
  if (!valid(c)) return 0;
  size_t total = 0;
  for (int l = 0; l < c->n_layers; ++l) {
    const size_t n_in_l = (l == 0) ? c->n_in : c->n_rec;
    const size_t n_pre = n_in_l + (c->recurrent ? c->n_rec : 0);
    const size_t N = c->n_rec, K = c->n_out;
    total += 2 * N * (c->fwd_fp32 ? sizeof(float) : sizeof(double));
    total += sizeof(double) * (2 * N + 2 * n_pre + N + 2 * K + N + K + N);
    total += sizeof(double) * N;   // last pseudo-derivative
    if (n_sample < 0)
      total += sizeof(double) * ((c->model == 1 ? 3 : c->reset_through ? 2 : 1) * N * n_pre +
                                 (size_t)c->n_adaptive * n_pre);
  }
  if (n_sample >= 0) total += sizeof(double) * (c->reset_through || c->model == 1 ? 3 : 2) * (size_t)n_sample;
  return total;
}

// Runs batch elements [b_lo, b_hi) over T steps and ADDS their gradient into
// the caller's fp64 buffers (zero them first to get dE/dW of those elements).
//   W[l]: [n_rec][n_pre_l] fp32 = [W_in | W_rec];  Wout[l]: [n_out][n_rec] fp32
//   x: [T][batch][n_in] bytes, nonzero = spike;  labels: [batch]
//   sample: NULL with n_sample < 0 for every synapse, dW[l] = [n_rec][n_pre_l];
//           else n_sample triples (layer, j, i) and dW[0] = [n_sample]
//   spikes: NULL or [T][n_layers][batch][ceil(n_rec/32)], bit j%32 of word j/32
//   dWout[l]: [n_out][n_rec];  loss: sum over b, t, layers of the cross-entropy
// Returns 0, or -1 on an invalid argument.
//   Fb: NULL, or per layer NULL or the feedback matrix B [n_out][n_rec] fp32
//       of the learning signal L = B^T delta (NULL: B = W_out).
int oracle_eprop_run_fb(const oracle_config* c, const float* const* W, const float* const* Wout,
                        const float* const* Fb, const uint8_t* x, int32_t T,
                        const int32_t* labels, int32_t b_lo, int32_t b_hi, const int32_t* sample,
                        int32_t n_sample, uint32_t* spikes, double* const* dW,
                        double* const* dWout, double* loss, const oracle_record* rec) {
  if (!valid(c) || !W || !Wout || !x || !labels || !dW || !dWout || !loss || T < 0 ||
      b_lo < 0 || b_hi > c->batch || b_lo > b_hi || (n_sample >= 0 && !sample))
    return -1;
  for (int b = b_lo; b < b_hi; ++b)
    if (labels[b] < 0 || labels[b] >= c->n_out) return -1;
  const Synapse* smp = reinterpret_cast<const Synapse*>(sample);
  for (int q = 0; q < n_sample; ++q) {
    const int l = smp[q].layer;
    if (l < 0 || l >= c->n_layers) return -1;
    const int n_pre = ((l == 0) ? c->n_in : c->n_rec) + (c->recurrent ? c->n_rec : 0);
    if (smp[q].j < 0 || smp[q].j >= c->n_rec || smp[q].i < 0 || smp[q].i >= n_pre) return -1;
  }
  if (c->fwd_fp32)
    return run<float>(*c, W, Wout, Fb, x, T, labels, b_lo, b_hi, smp, n_sample, spikes, dW, dWout,
                      loss, rec);
  return run<double>(*c, W, Wout, Fb, x, T, labels, b_lo, b_hi, smp, n_sample, spikes, dW, dWout,
                     loss, rec);
}

// Every batch element over T steps with online weight application every
// `every` steps (see run_online): dW, dWout (zeroed by the caller) receive the
// gradient of the whole run, W_final[l], Wout_final[l] (layouts of W, Wout)
// the weights in use at its end.  Spikes as oracle_eprop_run_fb; Fb as
// oracle_eprop_run_fb (NULL: the learning signal through the readout weights
// in use).
int oracle_eprop_run_online_fb(const oracle_config* c, const float* const* W,
                               const float* const* Wout, const float* const* Fb, const uint8_t* x,
                               int32_t T, const int32_t* labels, double lr, int32_t every,
                               uint32_t* spikes, double* const* dW, double* const* dWout,
                               double* loss, float* const* W_final, float* const* Wout_final) {
  if (!valid(c) || !W || !Wout || !x || !labels || !dW || !dWout || !loss || !W_final ||
      !Wout_final || T < 0 || every < 1)
    return -1;
  for (int b = 0; b < c->batch; ++b)
    if (labels[b] < 0 || labels[b] >= c->n_out) return -1;
  if (c->fwd_fp32)
    return run_online<float>(*c, W, Wout, Fb, x, T, labels, lr, every, spikes, dW, dWout, loss,
                             W_final, Wout_final);
  return run_online<double>(*c, W, Wout, Fb, x, T, labels, lr, every, spikes, dW, dWout, loss,
                            W_final, Wout_final);
}

int oracle_eprop_run_online(const oracle_config* c, const float* const* W,
                            const float* const* Wout, const uint8_t* x, int32_t T,
                            const int32_t* labels, double lr, int32_t every, uint32_t* spikes,
                            double* const* dW, double* const* dWout, double* loss,
                            float* const* W_final, float* const* Wout_final) {
  return oracle_eprop_run_online_fb(c, W, Wout, nullptr, x, T, labels, lr, every, spikes, dW, dWout,
                                    loss, W_final, Wout_final);
}

// The same with the learning signal through W_out (symmetric feedback).
int oracle_eprop_run(const oracle_config* c, const float* const* W, const float* const* Wout,
                     const uint8_t* x, int32_t T, const int32_t* labels, int32_t b_lo,
                     int32_t b_hi, const int32_t* sample, int32_t n_sample, uint32_t* spikes,
                     double* const* dW, double* const* dWout, double* loss,
                     const oracle_record* rec) {
  return oracle_eprop_run_fb(c, W, Wout, nullptr, x, T, labels, b_lo, b_hi, sample, n_sample,
                             spikes, dW, dWout, loss, rec);
}

}  // extern "C"
