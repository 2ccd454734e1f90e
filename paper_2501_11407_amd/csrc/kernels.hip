// gfx950 kernels of the online e-prop step.
//
// Built with -ffp-contract=off: every a*b+c written below is a rounded
// multiply followed by a rounded add unless fmaf/fma is spelled out.  The
// forward kernel relies on this to reproduce fp32 spike decisions operation
// by operation; the eligibility kernel uses explicit fused multiply-adds where
// precision only gains from them.
#include "kernels.h"

#include <math.h>

#include <algorithm>
#include <mutex>
#include <utility>

namespace eprop {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kSoftWave = kFwdWaves - 1;   // forward wave that runs the softmax

// Wave-wide reductions with DPP lane moves (no shared-memory round trip):
// within quads, half-rows and rows of 16 lanes, then across the four rows
// (row broadcasts of lanes 15 and 31); lane 63 ends with the result, which is
// returned to every lane.  Every lane must be active.
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_move(float v) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, ROWS, 0xF, false));
}
template <typename Op>
__device__ __forceinline__ float wave_reduce(float v, Op op) {
  v = op(v, dpp_move<0xB1, 0xF>(v));    // quad_perm [1,0,3,2]
  v = op(v, dpp_move<0x4E, 0xF>(v));    // quad_perm [2,3,0,1]
  v = op(v, dpp_move<0x141, 0xF>(v));   // row_half_mirror
  v = op(v, dpp_move<0x140, 0xF>(v));   // row_mirror
  v = op(v, dpp_move<0x142, 0xA>(v));   // row_bcast:15 into rows 1 and 3
  v = op(v, dpp_move<0x143, 0xC>(v));   // row_bcast:31 into rows 2 and 3
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
__device__ inline float wave_max(float v) {
  return wave_reduce(v, [](float a, float b) { return fmaxf(a, b); });
}
__device__ inline float wave_sum(float v) {
  return wave_reduce(v, [](float a, float b) { return a + b; });
}

__device__ inline int lanes_below(unsigned long long m, int lane) {
  return __popcll(m & ((1ull << lane) - 1ull));
}

inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

// Workgroup barrier for shared-memory data only: waits for this wave's LDS
// operations, not for its global stores (a __syncthreads fence would), which
// in the forward kernel are read only by later kernels.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0), vmcnt and expcnt unrestricted
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// ---------------------------------------------------------------- scaled fp16 pairs
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Power-of-two scale that puts a row's largest magnitude m in [2^13, 2^14)
// (exponent clamped for rows of tiny values); 0 for m == 0.
__device__ __forceinline__ int pair_exponent(float m) {
  if (!(m > 0.0f)) return 0;
  int k;
  (void)frexpf(m, &k);
  return min(100, max(-100, 14 - k));
}

// x (already scaled) -> hi = fp16(x), lo = fp16(x - hi)
__device__ __forceinline__ void split16(float x, _Float16& hi, _Float16& lo) {
  hi = (_Float16)x;
  lo = (_Float16)(x - (float)hi);
}

// 16 values x scale -> the 64-byte pair record of a chunk row: the 16 hi
// halves in step order (units 0 and 1), then the 16 lo halves (units 2, 3)
__device__ __forceinline__ void store_pairs(uint32_t* dst, const float (&x)[kChunk], float scale) {
  uint32_t h[kChunk / 2], l[kChunk / 2];
#pragma unroll
  for (int e = 0; e < kChunk; e += 2) {
    _Float16 h0, l0, h1, l1;
    split16(x[e] * scale, h0, l0);
    split16(x[e + 1] * scale, h1, l1);
    h[e / 2] = (uint32_t)__builtin_bit_cast(uint16_t, h0) | ((uint32_t)__builtin_bit_cast(uint16_t, h1) << 16);
    l[e / 2] = (uint32_t)__builtin_bit_cast(uint16_t, l0) | ((uint32_t)__builtin_bit_cast(uint16_t, l1) << 16);
  }
  u32x4* d = (u32x4*)dst;
  d[0] = u32x4{h[0], h[1], h[2], h[3]};
  d[1] = u32x4{h[4], h[5], h[6], h[7]};
  d[2] = u32x4{l[0], l[1], l[2], l[3]};
  d[3] = u32x4{l[4], l[5], l[6], l[7]};
}


// ---------------------------------------------------------------- forward
// One workgroup per batch element runs `steps` timesteps of every layer; the
// neuron state and, for each thread's own presynaptic rows, the filter, the
// chunk's p bits and the last spike stay in registers, the readout in shared
// memory.  Thread 64 w + l (wave
// w, lane l) holds the QN neurons 64 QN w + 64 q + l, q < QN (fwd_neuron): a
// wave owns a contiguous range of neurons, its spike list, built by ballots
// in ascending q, is ascending, and the waves' lists in wave order are the
// ascending list of the layer's spikes.  Per step and layer:
//   1. the active rows of p = [in ; z_prev] in ascending order: for the
//      first layer, the previous step's spike lists (its input rows enter
//      through the input drive, below); for a second layer, the first
//      layer's lists of this step and then its own of the previous step.
//   2. drive I_j: the first layer starts from its input drive, the sum of
//      W_ji over the step's active inputs in ascending i (input_drive_kernel;
//      it does not depend on the network state), a second layer from 0; the
//      listed rows are added in ascending i, so that I is the plain
//      sequential sum over the active rows.  While the rows' loads are in
//      flight: the filter zbar = alpha*zbar + p of the rows the workgroup
//      handles (recurrent rows, and every row of a second layer; the first
//      layer's input rows are input_filter_kernel's) and their p bits.  Then
//      the neuron step with one rounding per operation:
//        v = alpha*v; v = v + I; v = v - thr*z_prev
//        a = rho*a;   a = a + z_prev
//        A = beta_j*a; A = thr + A;  x = v - A;  z = x > 0
//        psi = (gamma/thr) * max(0, 1 - |x|/thr)
//   3. each wave sums the readout weights of its spiking neurons for every
//      class; ztilde = kappa*ztilde + z.
//   4. one wave: y = kappa*y + (sum of the waves' partial sums, in wave
//      order), softmax, delta = softmax - onehot(label), cross-entropy.
// The learning signal L = W_out^T delta is one GEMM over the whole block.
struct FwdLds {
  float* iring;                  // SVC: [3][512 QN] input drive of steps t, t+1, t+2 (slot t % 3)
  int* spk;                      // [n_layers][2][waves][jlist]: spike lists by step parity
  int* cnt;                      // [n_layers][2][waves]: their lengths
  int* nin;                      // [steps]: active inputs of the first layer per step
  float* part; float* sy;
  bool w16;                      // the int16 weights are exact (FwdLayer::W16)
  int w16max;                    // their largest |k|
};

// Per thread and layer, in registers: the spikes of the thread's neurons at
// the last step, and the filter (zbar) and current 16-step chunk's p bits
// (bit t % 16) of the presynaptic rows the thread owns: the recurrent rows
// of its neurons (slot q; a second layer's: slot QN + q) and, in a second
// layer, the input rows of the first layer's neurons it holds (slot q).  Every
// row the forward filters is owned this way, so the filter needs no shared
// memory.
template <int QN>
struct FwdRows {
  float zb[2 * QN];
  uint32_t bits[2 * QN];
  bool z[QN];
};

template <int QN>
__device__ __forceinline__ int fwd_neuron(int tid, int q) {
  return (tid >> 6) * (kWave * QN) + q * kWave + (tid & (kWave - 1));
}

// Softmax cross-entropy of one step for K_out <= 64, in one wave: lane k holds
// class k's output y (updated here) and gets delta_k = softmax_k - onehot_k.
// The waves' partial sums are added in wave order.
__device__ __forceinline__ float softmax_lanes(const FwdArgs& A, const float* part, float& y,
                                               int label, double& loss) {
  const int lane = threadIdx.x & (kWave - 1);
  const bool in = lane < A.K_out;
  // all partial sums read before any is used (lanes past K_out read class 0)
  const int kc = in ? lane : 0;
  float pw[kFwdWaves];
#pragma unroll
  for (int ww = 0; ww < kFwdWaves; ++ww) pw[ww] = part[ww * A.K_out + kc];
  float Y = 0.0f;
#pragma unroll
  for (int ww = 0; ww < kFwdWaves; ++ww) Y += pw[ww];
  float yy = A.kappa * y;
  yy = yy + Y;
  if (in) y = yy;
  const float m = wave_max(in ? yy : -INFINITY);
  const float ex = expf(in ? yy - m : -INFINITY);   // 0 past K_out
  const float se = wave_sum(ex);
  const bool label_ok = label >= 0 && label < A.K_out;
  const float yl = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(yy), label_ok ? label : 0));
  if (lane == 0) {
    if (label_ok)
      loss += (double)(logf(se) - (yl - m));
    else
      *A.err_flag = 1;
  }
  return ex / se - ((lane == label) ? 1.0f : 0.0f);
}

// Readout partial sums of the spikes of one step in one wave, K_out <= 64
// (lane k: class k): the rows of the transposed readout weights of the
// wave's spiking neurons (their list in spk), up to kReadoutRows loaded
// together, added in list order.
constexpr int kReadoutRows = 8;
struct ReadoutRows {
  float wv[kReadoutRows];
  int n;
};
__device__ __forceinline__ void readout_issue(const FwdArgs& A, const float* WoutT, const int* spk,
                                              int n_spk, ReadoutRows& R) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t koff = (uint32_t)min(lane, A.K_out - 1) * 4u;
  R.n = min(n_spk, kReadoutRows);
  const int ent = spk[min(lane & (kReadoutRows - 1), max(n_spk - 1, 0))];
#pragma unroll
  for (int u = 0; u < kReadoutRows; ++u) {
    const int j = __builtin_amdgcn_readlane(ent, u);
    R.wv[u] = u < R.n ? *(const float*)((const char*)(WoutT + (size_t)j * A.ldk) + koff) : 0.0f;
  }
}
__device__ __forceinline__ float readout_sum(const FwdArgs& A, const float* WoutT, const int* spk,
                                             int n_spk, const ReadoutRows& R) {
  const int lane = threadIdx.x & (kWave - 1);
  float Y = 0.0f;
#pragma unroll
  for (int u = 0; u < kReadoutRows; ++u)
    if (u < R.n) Y += R.wv[u];
  // more spikes in the wave (rare): the rest in further rounds
  const uint32_t koff = (uint32_t)min(lane, A.K_out - 1) * 4u;
  for (int s0 = kReadoutRows; s0 < n_spk; s0 += 16) {
    const int ent = spk[min(s0 + (lane & 15), n_spk - 1)];
    float wv[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int j = __builtin_amdgcn_readlane(ent, u);
      wv[u] = *(const float*)((const char*)(WoutT + (size_t)j * A.ldk) + koff);
    }
#pragma unroll
    for (int u = 0; u < 16; ++u)
      if (s0 + u < n_spk) Y += wv[u];
  }
  return Y;
}

// The spike list of a wave (parity par) from its neurons' spikes, for the
// block's first step; returns its length.
template <int QN, int LI>
__device__ __forceinline__ int wave_list_from_regs(const FwdArgs& A, const FwdLds& S, int par,
                                                   const FwdRows<QN>& R) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  int* spk = S.spk + ((LI * 2 + par) * kFwdWaves + w) * A.jlist;
  int n = 0;
#pragma unroll
  for (int q = 0; q < QN; ++q) {
    const int j = fwd_neuron<QN>(tid, q);
    const bool z = j < A.n_rec && R.z[q];
    const unsigned long long m = __ballot(z);
    if (z) spk[n + lanes_below(m, lane)] = j;
    n += __popcll(m);
  }
  if (lane == 0) S.cnt[(LI * 2 + par) * kFwdWaves + w] = n;
  return n;
}

// A buffer resource over [base, base + bytes): loads past the range read
// zero and stores past it write nothing.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}

// SOFTWIN: the softmax runs while the drive's loads are in flight (else at
// the step's start, which needs fewer registers at the loads).  SVC: the
// input drive comes from the shared-memory ring the service wave fills
// (else each thread loads the next step's itself).
// R: this layer's rows and spikes; R0: the first layer's (a second layer's
// input: its spikes of this step).
template <int QN, int LI, bool SOFTWIN, bool SVC>
__device__ __forceinline__ void forward_layer_step(const FwdArgs& A, const FwdLds& S, int t, int b,
                                                   float (&v)[QN], float (&ad)[QN],
                                                   float (&zt)[QN], double& loss, int label,
                                                   float& yk, float& dk, int& nspk_prev,
                                                   float (&iin)[QN], FwdRows<QN>& R,
                                                   const FwdRows<QN>& R0) {
  const FwdLayer& Ly = A.L[LI];
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const bool recurrent = Ly.n_pre > Ly.n_inl;
  float* sy = S.sy + LI * A.K_out;
  const int pc = t & 1, pp = pc ^ 1;           // parity of this and the previous step
  int* spk_now = S.spk + ((LI * 2 + pc) * kFwdWaves + w) * A.jlist;
  const int* spk_prev = S.spk + ((LI * 2 + pp) * kFwdWaves + w) * A.jlist;
  const size_t row = (size_t)t * A.Bp + b;
  // readout partial sums by step parity
  float* part = S.part + (LI * 2 + pc) * kFwdWaves * A.K_out;
  // K_out <= 64: the readout of a step's spikes is loaded together with the
  // next step's drive (its partial sums go to part of that step's parity),
  // and the softmax of the step two back is taken during this step, by the
  // service wave where there is one (SVC), else by the last wave, which
  // stores delta with this step's stores; the block's last two steps are
  // finished after the step loop
  const bool defer = A.K_out <= kWave;
  constexpr bool SOFTHERE = !SVC;   // this wave group takes the deferred softmax
  if (SOFTHERE && !SOFTWIN && defer && w == kSoftWave && t > 1) dk = softmax_lanes(A, part, yk, label, loss);

  // 1. the active rows: segments of spike lists (LDS int offsets), each with
  // the row index of its neuron 0
  constexpr int NSEG = LI == 0 ? kFwdWaves : 2 * kFwdWaves;
  int offs[NSEG];
  int total = 0;
  {
    const int* c0 = S.cnt + (LI == 0 ? (0 * 2 + pp) : (0 * 2 + pc)) * kFwdWaves;
    const int* c1 = S.cnt + (1 * 2 + pp) * kFwdWaves;
    // the first segments: a second layer's inputs, or the first layer's
    // recurrent rows (none in a feed-forward layer)
    int cl = 0;
    if (lane < kFwdWaves && (LI == 1 || recurrent)) cl = c0[lane];
    else if (LI == 1 && recurrent && lane >= kFwdWaves && lane < 2 * kFwdWaves) cl = c1[lane - kFwdWaves];
#pragma unroll
    for (int s = 0; s < NSEG; ++s) {
      offs[s] = total;
      total += __builtin_amdgcn_readlane(cl, s);
    }
  }
  const int seg0 = (LI == 0 ? (0 * 2 + pp) : (0 * 2 + pc)) * kFwdWaves * A.jlist;
  const int seg1 = (1 * 2 + pp) * kFwdWaves * A.jlist;
  const int roff0 = LI == 0 ? Ly.n_inl : 0;    // row of neuron 0 in the first segments
  auto list_entry = [&](int e) {
    int s = 0, o = 0;
#pragma unroll
    for (int u = 1; u < NSEG; ++u)
      if (e >= offs[u]) {
        s = u;
        o = offs[u];
      }
    const bool hi = LI == 1 && s >= kFwdWaves;
    const int base = hi ? seg1 + (s - kFwdWaves) * A.jlist : seg0 + s * A.jlist;
    return S.spk[base + (e - o)] + (hi ? A.n_rec : roff0);
  };
  const int zslot = t & (kChunk - 1);
  auto filter_one = [&](int k, bool on) {
    if (on) R.bits[k] |= 1u << zslot;
    R.zb[k] = A.alpha * R.zb[k] + (on ? 1.0f : 0.0f);
  };
  // The presynaptic filter and the next step's input drive, off the
  // critical path: issued while the drive's loads are in flight.
  float inext[QN];
#pragma unroll
  for (int q = 0; q < QN; ++q) inext[q] = 0.0f;
  bool filtered = false;
  auto filter_rows = [&]() {
    if (filtered) return;
    filtered = true;
    if (SOFTHERE && SOFTWIN && defer && w == kSoftWave && t > 1) dk = softmax_lanes(A, part, yk, label, loss);
    if constexpr (LI == 0 && !SVC) {
      if (t + 1 < A.steps) {
        typedef float fqv __attribute__((ext_vector_type(QN)));
        const fqv nv = *(const fqv*)(A.Iin + ((size_t)(t + 1) * A.B + b) * (QN * kFwdThreads) +
                                     (size_t)tid * QN);
#pragma unroll
        for (int q = 0; q < QN; ++q) inext[q] = nv[q];
      }
    }
#pragma unroll
    for (int q = 0; q < QN; ++q) {
      if (fwd_neuron<QN>(tid, q) >= A.n_rec) continue;
      if (LI == 0) {
        if (recurrent) filter_one(q, R.z[q]);
      } else {
        filter_one(q, R0.z[q]);
        if (recurrent) filter_one(QN + q, R.z[q]);
      }
    }
  };

  // 2. drive and neuron step.  UB rows are loaded before any is added: lane
  // u reads list entry k0 + u, every wave takes the entries from its lanes,
  // and each row's load is a scalar row base plus the lane offset.
  constexpr int UB = QN >= 16 ? 1 : 16 / QN;
  // the readout rows of the previous step's spikes, loaded with the drive rows
  ReadoutRows rr;
  if (defer && t > 0) readout_issue(A, Ly.WoutT, spk_prev, nspk_prev, rr);
  float I[QN];
  if constexpr (LI == 0 && SVC) {
    typedef float fqv __attribute__((ext_vector_type(QN)));
    const fqv rv = *(const fqv*)(S.iring + (t % 3) * (QN * kFwdThreads) + tid * QN);
#pragma unroll
    for (int q = 0; q < QN; ++q) I[q] = rv[q];
  } else {
#pragma unroll
    for (int q = 0; q < QN; ++q) I[q] = LI == 0 ? iin[q] : 0.0f;
  }
  // integer weights k (w = k 2^-14, |k| <= 32767): with at most 2^24 / max|k|
  // active rows every partial sum in any order is an integer of at most
  // 2^24 units, exact in fp32, so the integer sum plus the (then exact)
  // input drive equals the fp32 sequential sum; decided per step from the
  // step's active rows, inputs included
  const int all_rows = total + (LI == 0 ? S.nin[t] : 0);
  const bool w16 = S.w16 && (long long)all_rows * S.w16max <= (1ll << 24);
  if (w16) {
    // the thread's QN of a row in one load of 2 QN bytes
    constexpr int UB16 = QN <= 2 ? 16 : 32 / QN;
    typedef int16_t i16v __attribute__((ext_vector_type(QN)));
    int isum[QN];
#pragma unroll
    for (int q = 0; q < QN; ++q) isum[q] = 0;
    // A batch's entries past the list get row n_pre, a row of zeros after
    // the layer's rows, so every load and every add is unconditional (no
    // branch per row) and the integer sum is unchanged.  Each load is the
    // row base plus a 32-bit per-lane offset.
    const char* w16 = (const char*)Ly.W16;
    const uint32_t voff = (uint32_t)tid * (QN * 2);
    for (int k0 = 0; k0 < total; k0 += UB16) {
      const int e = k0 + (lane & (UB16 - 1));
      const int le = list_entry(min(e, total - 1));
      const int ent = e < total ? le : Ly.n_pre;
      i16v wk[UB16];
#pragma unroll
      for (int u = 0; u < UB16; ++u) {
        const uint32_t i = (uint32_t)__builtin_amdgcn_readlane(ent, u);
        wk[u] = *(const i16v*)(w16 + (voff + i * (uint32_t)(QN * kFwdThreads * 2)));
      }
      __builtin_amdgcn_sched_barrier(0);
      filter_rows();
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < UB16; ++u)
#pragma unroll
        for (int q = 0; q < QN; ++q) isum[q] += (int)wk[u][q];
    }
#pragma unroll
    for (int q = 0; q < QN; ++q) I[q] = I[q] + (float)isum[q] * 0x1p-14f;
  }
  // fp32 rows: the same scheme (entries past the list read the zero row
  // n_pre); the zeros are added after every listed row, to a sum that is
  // never -0 (it starts at +0 and a sum of opposite values rounds to +0), so
  // the sum's bits are those of the listed rows' sequential sum
  const char* wt = (const char*)Ly.Wt;
  for (int k0 = 0; !w16 && k0 < total; k0 += UB) {
    const int e = k0 + (lane & (UB - 1));
    const int le = list_entry(min(e, total - 1));
    const int ent = e < total ? le : Ly.n_pre;
    float wv[UB][QN];
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const uint32_t i = (uint32_t)__builtin_amdgcn_readlane(ent, u);
#pragma unroll
      for (int q = 0; q < QN; ++q)
        wv[u][q] = *(const float*)(wt + (i * (uint32_t)Ly.ldw + (uint32_t)fwd_neuron<QN>(tid, q)) * 4u);
    }
    __builtin_amdgcn_sched_barrier(0);
    filter_rows();
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < UB; ++u)
#pragma unroll
      for (int q = 0; q < QN; ++q) I[q] += wv[u][q];
  }
  filter_rows();   // (no active row this step)
  if (defer && t > 0) {
    const float Y = readout_sum(A, Ly.WoutT, spk_prev, nspk_prev, rr);
    float* part_prev = S.part + (LI * 2 + pp) * kFwdWaves * A.K_out;
    if (lane < A.K_out) part_prev[w * A.K_out + lane] = Y;
  }
  int n_spk = 0;
  float psv[QN];
  unsigned long long smask[QN];
#pragma unroll
  for (int q = 0; q < QN; ++q) {
    const int j = fwd_neuron<QN>(tid, q);
    bool z = false;
    psv[q] = 0.0f;
    if (j < A.n_rec) {
      const float zp = R.z[q] ? 1.0f : 0.0f;
      float x;
      if (A.model == 1) {
        // a step linear in its two state components with host-derived
        // coefficients (the two-compartment neuron: h0 soma, h1 dendrite),
        // each component summed in the order A h_prev, b I, r z_prev
        float h1 = A.mA[1][0] * v[q];
        h1 = h1 + A.mA[1][1] * ad[q];
        h1 = h1 + A.mb[1] * I[q];
        h1 = h1 + A.mr[1] * zp;
        float h0 = A.mA[0][0] * v[q];
        h0 = h0 + A.mA[0][1] * ad[q];
        h0 = h0 + A.mb[0] * I[q];
        h0 = h0 + A.mr[0] * zp;
        float u = A.mc[0] * h0;
        u = u + A.mc[1] * h1;
        x = u - A.thr;
        v[q] = h0;
        ad[q] = h1;
      } else {
        float vv = A.alpha * v[q];
        vv = vv + I[q];
        vv = vv - A.thr * zp;
        float aa = A.rho * ad[q];
        aa = aa + zp;
        const float bj = (j < A.n_adaptive) ? A.beta : 0.0f;
        float th = bj * aa;
        th = A.thr + th;
        x = vv - th;
        v[q] = vv;
        ad[q] = aa;
      }
      z = x > 0.0f;
      R.z[q] = z;
      // |x|/thr as a product with 1/thr (the same value for a power-of-two
      // threshold; within a rounding of it otherwise, and psi only enters
      // the gradient)
      const float u = 1.0f - fabsf(x) * A.inv_thr;
      psv[q] = A.gamma_over_thr * fmaxf(u, 0.0f);
      float zz = A.kappa * zt[q];
      zz = zz + (z ? 1.0f : 0.0f);
      zt[q] = zz;
    }
    const unsigned long long m = __ballot(z);
    smask[q] = m;
    if (z) spk_now[n_spk + lanes_below(m, lane)] = j;
    n_spk += __popcll(m);
  }
  if (lane == 0) S.cnt[(LI * 2 + pc) * kFwdWaves + w] = n_spk;
  nspk_prev = n_spk;
  if constexpr (LI == 0 && !SVC) {
#pragma unroll
    for (int q = 0; q < QN; ++q) iin[q] = inext[q];
  }

  // 3. (K_out > 64) this wave's share of the readout: rows of the transposed
  // readout weights of its spiking neurons, read coalesced over the classes
  for (int kb = 0; !defer && kb < A.K_out; kb += kWave) {
    const int k = kb + lane;
    const uint32_t koff = (uint32_t)min(k, A.K_out - 1) * 4u;
    float Y = 0.0f;
    for (int s0 = 0; s0 < n_spk; s0 += 16) {
      const int ent = spk_now[min(s0 + (lane & 15), n_spk - 1)];
      float wv[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int j = __builtin_amdgcn_readlane(ent, u);
        wv[u] = *(const float*)((const char*)(Ly.WoutT + (size_t)j * A.ldk) + koff);
      }
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (s0 + u < n_spk) Y += wv[u];
    }
    if (k < A.K_out) part[w * A.K_out + k] = Y;
  }

  // Global stores of the step go last: a load waits for every store issued
  // before it, so stores ahead of the drive and readout loads would lengthen
  // the step.  Per-step vectors: psi, ztilde, the spike words, and (every
  // 16 steps) the binary presynaptic bits ([b][t/16][i]).
#pragma unroll
  for (int q = 0; q < QN; ++q) {
    const int j = fwd_neuron<QN>(tid, q);
    if (j < A.n_rec) {
      __builtin_nontemporal_store(psv[q], Ly.psiK + row * A.ldj + j);
      __builtin_nontemporal_store(zt[q], Ly.ztK + row * A.ldn + j);
    }
    if (A.spikes) {
      const int w0 = (w * (kWave * QN) + q * kWave) >> 5;
      uint32_t* srow = A.spikes + (((size_t)t * A.n_layers + LI) * A.B + b) * A.W32;
      if (lane == 0 && w0 < A.W32) __builtin_nontemporal_store((uint32_t)smask[q], srow + w0);
      if (lane == 1 && w0 + 1 < A.W32) __builtin_nontemporal_store((uint32_t)(smask[q] >> 32), srow + w0 + 1);
    }
  }
  if (SOFTHERE && defer && w == kSoftWave && t > 1 && lane < A.K_out)
    __builtin_nontemporal_store(dk, Ly.deltaK + (row - 2 * A.Bp) * A.ldk + lane);
  // the p bits of a chunk go out at its last step (or the block's), one
  // 16-bit word per row, and the row's bits start over (bits past the
  // block's last step are zero)
  if ((t & (kChunk - 1)) == kChunk - 1 || t == A.steps - 1) {
    uint16_t* cb = Ly.pbits + ((size_t)b * kKC + t / kChunk) * Ly.ldi;
    auto flush = [&](int k, int i) {
      __builtin_nontemporal_store((uint16_t)R.bits[k], cb + i);
      R.bits[k] = 0u;
    };
#pragma unroll
    for (int q = 0; q < QN; ++q) {
      const int j = fwd_neuron<QN>(tid, q);
      if (j >= A.n_rec) continue;
      if (LI == 0) {
        if (recurrent) flush(q, Ly.n_inl + j);
      } else {
        flush(q, j);
        if (recurrent) flush(QN + q, A.n_rec + j);
      }
    }
  }
  lds_barrier();

  // 4. readout, softmax cross-entropy (K_out > 64; the other waves go on)
  if (!defer && w == kSoftWave) {
    const bool label_ok = label >= 0 && label < A.K_out;
    float m = -INFINITY;
    for (int k = lane; k < A.K_out; k += kWave) {
      float Y = 0.0f;
      for (int ww = 0; ww < kFwdWaves; ++ww) Y += part[ww * A.K_out + k];
      float yy = A.kappa * sy[k];
      yy = yy + Y;
      sy[k] = yy;
      m = fmaxf(m, yy);
    }
    m = wave_max(m);
    float se = 0.0f;
    for (int k = lane; k < A.K_out; k += kWave) se += expf(sy[k] - m);
    se = wave_sum(se);
    if (lane == 0) {
      if (label_ok)
        loss += (double)(logf(se) - (sy[label] - m));
      else
        *A.err_flag = 1;
    }
    for (int k = lane; k < A.K_out; k += kWave) {
      const float d = expf(sy[k] - m) / se - ((k == label) ? 1.0f : 0.0f);
      Ly.deltaK[row * A.ldk + k] = d;
    }
  }
}

// The state of one layer in (load) or out.  The filter rows are those the
// workgroup handles (ridx.. in shared memory, presynaptic rows i0.. of the
// layer); on load the filter also goes to zstart for the eligibility pass.
template <int QN, int LI>
__device__ __forceinline__ void forward_state(const FwdArgs& A, const FwdLds& S, int b, bool load,
                                              float (&v)[QN], float (&ad)[QN], float (&zt)[QN],
                                              FwdRows<QN>& R) {
  const FwdLayer& Ly = A.L[LI];
  const int tid = threadIdx.x;
  float* sy = S.sy + LI * A.K_out;
  const bool recurrent = Ly.n_pre > Ly.n_inl;
  // the filter of row i (load: also the block-start filter zstart)
  auto row = [&](int k, int i) {
    float* zb = Ly.zbar + (size_t)b * Ly.n_pre + i;
    if (load) {
      R.zb[k] = *zb;
      R.bits[k] = 0u;
      Ly.zstart[(size_t)b * Ly.ldi + i] = R.zb[k];
    } else {
      *zb = R.zb[k];
    }
  };
#pragma unroll
  for (int q = 0; q < QN; ++q) {
    const int j = fwd_neuron<QN>(tid, q);
    if (j < A.n_rec) {
      const size_t o = (size_t)b * A.n_rec + j;
      if (load) {
        v[q] = Ly.v[o]; ad[q] = Ly.a[o]; zt[q] = Ly.ztil[o]; R.z[q] = Ly.z[o] != 0;
      } else {
        Ly.v[o] = v[q]; Ly.a[o] = ad[q]; Ly.ztil[o] = zt[q]; Ly.z[o] = R.z[q] ? 1 : 0;
      }
      if (LI == 0) {
        if (recurrent) row(q, Ly.n_inl + j);
      } else {
        row(q, j);
        if (recurrent) row(QN + q, A.n_rec + j);
      }
    }
  }
  for (int k = tid; k < A.K_out; k += kFwdThreads) {
    if (load) sy[k] = Ly.y[(size_t)b * A.K_out + k];
    else Ly.y[(size_t)b * A.K_out + k] = sy[k];
  }
}

// The service wave (SVC): a ninth wave that owns no neurons.  During step t
// it writes the input drive of step t + 2 into ring slot (t + 2) % 3 (read by
// the other waves at step t + 2; its last reader, step t - 1, is past the
// barrier) from registers loaded during step t - 1, then loads step t + 3's.
// Its global loads are its own: the vector-memory counter is per wave, so the
// other waves' waits for their drive rows never include them.  It takes part
// in every barrier of the workgroup.
template <int QN, int NL>
__device__ __forceinline__ void forward_service_wave(const FwdArgs& A, const FwdLds& S, int b) {
  constexpr int NV = QN * kFwdThreads / (4 * kWave);   // 16-byte vectors per lane and step
  const int l = threadIdx.x & (kWave - 1);
  f32x4 R[NV];
  auto load = [&](int tt) {
    const float* src = A.Iin + ((size_t)tt * A.B + b) * (QN * kFwdThreads);
#pragma unroll
    for (int k = 0; k < NV; ++k) R[k] = *(const f32x4*)(src + k * 4 * kWave + 4 * l);
  };
  auto put = [&](int slot) {
    float* d = S.iring + slot * (QN * kFwdThreads);
#pragma unroll
    for (int k = 0; k < NV; ++k) *(f32x4*)(d + k * 4 * kWave + 4 * l) = R[k];
  };
  for (int tt = 0; tt < min(2, A.steps); ++tt) {
    load(tt);
    put(tt);
  }
  if (A.steps > 2) load(2);
  // K_out <= 64: the deferred softmax (lane k: class k), off the compute
  // waves' path: during step t, that of step t - 2 of every layer (its
  // partial sums are complete since the end of step t - 1 and are next
  // overwritten in step t + 1), delta stored for that step; y (the readout
  // filter) in registers from the block's start to its end; the loss added
  // to the batch element's sum at the end
  const bool defer = A.K_out <= kWave;
  const int label = __builtin_amdgcn_readfirstlane(A.labels[b]);
  float y[NL];
  double loss[NL];
  lds_barrier();                                   // the others' barrier before the step loop
#pragma unroll
  for (int li = 0; li < NL; ++li) {
    y[li] = l < A.K_out ? S.sy[li * A.K_out + l] : 0.0f;
    loss[li] = 0.0;
  }
  auto softmax_step = [&](int ts) {
#pragma unroll
    for (int li = 0; li < NL; ++li) {
      const float d = softmax_lanes(A, S.part + (li * 2 + (ts & 1)) * kFwdWaves * A.K_out, y[li], label,
                                    loss[li]);
      if (l < A.K_out)
        __builtin_nontemporal_store(d, A.L[li].deltaK + ((size_t)ts * A.Bp + b) * A.ldk + l);
    }
  };
  for (int t = 0; t < A.steps; ++t) {
    if (t + 2 < A.steps) {
      put((t + 2) % 3);
      if (t + 3 < A.steps) load(t + 3);
    }
    if (defer && t > 1) softmax_step(t - 2);
    for (int li = 0; li < NL; ++li) lds_barrier();   // one per layer step
  }
  if (defer && A.steps > 0) {
    lds_barrier();                                 // the last readout
    for (int ts = max(A.steps - 2, 0); ts < A.steps; ++ts) softmax_step(ts);
    if (l < A.K_out)
#pragma unroll
      for (int li = 0; li < NL; ++li) S.sy[li * A.K_out + l] = y[li];
    if (l == 0)
#pragma unroll
      for (int li = 0; li < NL; ++li) A.L[li].lossacc[b] += loss[li];
  }
  lds_barrier();                                   // before the state goes out
}

// Four waves per SIMD (128 registers) for one layer of at most two neurons
// per thread; three (168) for two layers or four neurons per thread and
// more, so that those do not spill up to four.  An eligibility workgroup
// (168 registers per wave) fits beside the forward on its compute unit where
// the forward's waves per SIMD times their registers leave 168: one layer of
// at most two neurons per thread or two of one (nine waves, three on one
// SIMD, at most 112 registers), and every form without the service wave
// (eight waves, two per SIMD).
template <int QN, int NL, bool SVC>
__global__ __launch_bounds__(SVC ? kFwdThreads + 64 : kFwdThreads) __attribute__((amdgpu_waves_per_eu((QN >= 4 || NL > 1) ? 3 : 4))) void forward_kernel(FwdArgs A) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  // the forward is the sequential part of the step: its waves win instruction
  // issue over the eligibility waves that share their compute units
  __builtin_amdgcn_s_setprio(3);
  const int b = blockIdx.x;
  FwdLds S;
  S.iring = (float*)smem;                          // SVC: [3][512 QN]
  S.spk = (int*)(S.iring + (SVC ? 3 * QN * kFwdThreads : 0));   // [NL][2][waves][jlist]
  S.cnt = S.spk + NL * 2 * kFwdWaves * A.jlist;    // [NL][2][waves]
  S.nin = S.cnt + NL * 2 * kFwdWaves;              // [Kmax]
  S.part = (float*)(S.nin + A.Kmax);               // [NL][2][waves][K_out]
  S.sy = S.part + NL * 2 * kFwdWaves * A.K_out;    // [NL][K_out]
  S.w16 = A.w16ok[0] != 0;
  S.w16max = A.w16ok[1];
  if constexpr (SVC) {
    if (threadIdx.x >= kFwdThreads) {
      forward_service_wave<QN, NL>(A, S, b);
      return;
    }
  }

  for (int e = threadIdx.x; e < A.steps; e += kFwdThreads) S.nin[e] = A.nin[(size_t)e * A.B + b];
  float v0[QN], a0[QN], zt0[QN], v1[QN], a1[QN], zt1[QN];
  FwdRows<QN> R0, R1;
  forward_state<QN, 0>(A, S, b, true, v0, a0, zt0, R0);
  if constexpr (NL > 1) forward_state<QN, 1>(A, S, b, true, v1, a1, zt1, R1);
  // the spike lists of the step before the block (parity 1), from the
  // spikes each thread has just loaded for its own neurons
  wave_list_from_regs<QN, 0>(A, S, 1, R0);
  if constexpr (NL > 1) wave_list_from_regs<QN, 1>(A, S, 1, R1);
  double loss0 = 0.0, loss1 = 0.0;
  // loaded once: a global load inside the step would wait for the step's stores
  const int label = __builtin_amdgcn_readfirstlane(A.labels[b]);
  // the first step's input drive (with the service wave: in the ring)
  float iin[QN];
  if constexpr (!SVC) {
    typedef float fqv __attribute__((ext_vector_type(QN)));
    const fqv nv = *(const fqv*)(A.Iin + (size_t)b * (QN * kFwdThreads) + (size_t)threadIdx.x * QN);
#pragma unroll
    for (int q = 0; q < QN; ++q) iin[q] = nv[q];
  }
  lds_barrier();
  // deferred softmax state (the softmax wave, lane k: class k)
  const int lane = threadIdx.x & (kWave - 1);
  float y0 = 0.0f, y1 = 0.0f, d0 = 0.0f, d1 = 0.0f;
  if (lane < A.K_out) {
    y0 = S.sy[lane];
    if constexpr (NL > 1) y1 = S.sy[A.K_out + lane];
  }
  // spikes of the previous step in this wave whose readout is still to be
  // summed, per layer (none at the block's start)
  int ns0 = 0, ns1 = 0;
  float unused[QN];
  for (int t = 0; t < A.steps; ++t) {
    // two layers of four neurons per thread and more: the softmax at the
    // step's start (no spills)
    constexpr bool SW = NL == 1 || QN < 4;
    forward_layer_step<QN, 0, SW, SVC>(A, S, t, b, v0, a0, zt0, loss0, label, y0, d0, ns0, iin, R0, R0);
    if constexpr (NL > 1)
      forward_layer_step<QN, 1, SW, SVC>(A, S, t, b, v1, a1, zt1, loss1, label, y1, d1, ns1, unused, R1, R0);
  }
  if (A.K_out <= kWave && A.steps > 0) {
    // the readout of the last step's spikes, then the softmax of the last
    // two steps (every step ends with a barrier, so the partial sums of the
    // step before the last are visible)
    const int tl = A.steps - 1;
    const int w = threadIdx.x >> 6;
    auto last_readout = [&](int li, int ns) {
      const float* WoutT = li == 0 ? A.L[0].WoutT : A.L[1].WoutT;
      const int* spk = S.spk + ((li * 2 + (tl & 1)) * kFwdWaves + w) * A.jlist;
      ReadoutRows rr;
      readout_issue(A, WoutT, spk, ns, rr);
      const float Y = readout_sum(A, WoutT, spk, ns, rr);
      if (lane < A.K_out) S.part[((li * 2 + (tl & 1)) * kFwdWaves + w) * A.K_out + lane] = Y;
    };
    last_readout(0, ns0);
    if constexpr (NL > 1) last_readout(1, ns1);
    lds_barrier();
    if (!SVC && w == kSoftWave) {
      for (int ts = max(tl - 1, 0); ts <= tl; ++ts) {
        const size_t row = (size_t)ts * A.Bp + b;
        d0 = softmax_lanes(A, S.part + (ts & 1) * kFwdWaves * A.K_out, y0, label, loss0);
        if (lane < A.K_out) __builtin_nontemporal_store(d0, A.L[0].deltaK + row * A.ldk + lane);
        if constexpr (NL > 1) {
          d1 = softmax_lanes(A, S.part + (2 + (ts & 1)) * kFwdWaves * A.K_out, y1, label, loss1);
          if (lane < A.K_out) __builtin_nontemporal_store(d1, A.L[1].deltaK + row * A.ldk + lane);
        }
      }
      if (lane < A.K_out) {
        S.sy[lane] = y0;
        if constexpr (NL > 1) S.sy[A.K_out + lane] = y1;
      }
    }
  }
  lds_barrier();
  forward_state<QN, 0>(A, S, b, false, v0, a0, zt0, R0);
  if constexpr (NL > 1) forward_state<QN, 1>(A, S, b, false, v1, a1, zt1, R1);
  // lane 0 of the softmax wave holds the loss (with the deferred softmax in
  // the service wave: that wave's, added there)
  if (threadIdx.x == kSoftWave * kWave && (!SVC || A.K_out > kWave)) {
    A.L[0].lossacc[b] += loss0;
    if constexpr (NL > 1) A.L[1].lossacc[b] += loss1;
  }
}

// ---------------------------------------------------------------- input drive and filter
// The rows listed in lst[0, n) (ascending input indices) added to acc in
// that order, U rows loaded before any is added: int16 rows kept packed
// until the add (exact: the same values as Wt), fp32 rows from Wt at the
// lane's neurons jof.
template <int PW, bool W16>
__device__ __forceinline__ void add_input_rows(const InputArgs& a, const int* lst, int n, int p0,
                                               const int (&jof)[PW], float (&acc)[PW]) {
  constexpr int U = W16 ? 8 : 4;
  const int lane = threadIdx.x & (kWave - 1);
  const int qnp = a.qn * kFwdThreads;
  for (int k0 = 0; k0 < n; k0 += U) {
    const int ent = lst[min(k0 + (lane & (U - 1)), n - 1)];
    const int nb = min(U, n - k0);   // rows of this batch (wave-uniform)
    if constexpr (W16) {
      typedef int16_t i16p __attribute__((ext_vector_type(PW)));
      i16p k[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = __builtin_amdgcn_readlane(ent, u);
        if (u < nb) k[u] = *(const i16p*)(a.W16 + (size_t)r * qnp + p0);
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (u < nb)
#pragma unroll
          for (int e = 0; e < PW; ++e) acc[e] = acc[e] + (float)k[u][e] * 0x1p-14f;
    } else {
      float wr[U][PW];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int r = __builtin_amdgcn_readlane(ent, u);
        if (u < nb)
#pragma unroll
          for (int e = 0; e < PW; ++e) wr[u][e] = a.Wt[(size_t)r * a.ldw + jof[e]];
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (u < nb)
#pragma unroll
          for (int e = 0; e < PW; ++e) acc[e] = acc[e] + wr[u][e];
    }
  }
}

// The first layer's input part of the drive for every step of a block, one
// wave per (step, batch element) and slice of 64 PW forward positions: the
// active inputs in ascending order, listed in shared memory (up to kInList
// at a time), their rows added in that order in fp32 starting from 0, the
// prefix of the forward's sequential sum.  Rows come from W16 (exact: the
// same values) when *w16ok, else from Wt.  Also the number of active
// inputs.  Input rows whose length is a multiple of 4 are read as 32-bit
// words, 1024 inputs per round trip (lane l holds inputs 4 l .. 4 l + 3 of
// each 256); other rows as bytes, 512 per round trip.
constexpr int kInPW = 8;     // forward positions per lane
constexpr int kInList = 256; // list entries per wave
__global__ __launch_bounds__(256) void input_drive_kernel(InputArgs a) {
  constexpr int PW = kInPW;
  __shared__ int lists[4][kInList];
  const int lane = threadIdx.x & (kWave - 1);
  int* lst = lists[threadIdx.x >> 6];
  const int wv = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int qsh = __builtin_ctz(a.qn);                // qn is a power of two
  const int slices = a.qn;                            // 512 qn / (64 PW)
  const int pair = wv >> qsh;
  if (pair >= a.steps * a.B) return;                  // the whole wave (no barriers below)
  const int sl = wv & (slices - 1);
  const int t = pair / a.B, b = pair - t * a.B;
  const uint8_t* xr = a.x + ((size_t)t * a.B + b) * a.n_in;
  const int p0 = (sl * kWave + lane) * PW;            // the lane's first position
  const bool w16 = a.w16ok[0] != 0;
  // the neurons of the lane's positions (position tid*QN + q holds neuron
  // 64 QN (tid / 64) + 64 q + tid % 64), for rows of Wt
  int jof[PW];
#pragma unroll
  for (int e = 0; e < PW; ++e) {
    const int p = p0 + e, tid = p >> qsh, q = p & (a.qn - 1);
    jof[e] = ((tid >> 6) << (6 + qsh)) + q * kWave + (tid & (kWave - 1));
  }
  float acc[PW];
#pragma unroll
  for (int e = 0; e < PW; ++e) acc[e] = 0.0f;
  auto flush = [&](int n) {
    if (w16) add_input_rows<PW, true>(a, lst, n, p0, jof, acc);
    else add_input_rows<PW, false>(a, lst, n, p0, jof, acc);
  };
  int cnt = 0, n = 0;   // active inputs so far; entries in the list
  const bool words = (a.n_in & 3) == 0 && ((uintptr_t)a.x & 3) == 0;
  if (words) {
    constexpr int G = 4;   // words per lane loaded together
    const int nw = a.n_in >> 2;
    const uint32_t* xw = (const uint32_t*)xr;
    for (int base = 0; base < nw; base += kWave * G) {
      uint32_t xv[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int k = base + g * kWave + lane;
        xv[g] = k < nw ? xw[k] : 0u;
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        unsigned long long m[4];
        int below = 0, c = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          m[k] = __ballot(((xv[g] >> (8 * k)) & 0xFFu) != 0);
          below += lanes_below(m[k], lane);
          c += __popcll(m[k]);
        }
        if (n + c > kInList) {   // the list is full: add its rows first
          flush(n);
          n = 0;
        }
        int own = 0;
        const int i0 = 4 * (base + g * kWave + lane);
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if ((xv[g] >> (8 * k)) & 0xFFu) lst[n + below + own++] = i0 + k;
        n += c;
        cnt += c;
      }
    }
  } else {
    constexpr int G = 8;   // bytes per lane loaded together
    for (int base = 0; base < a.n_in; base += kWave * G) {
      uint8_t xv[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int i = base + g * kWave + lane;
        xv[g] = i < a.n_in ? xr[i] : 0;
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const bool on = xv[g] != 0;
        const unsigned long long m = __ballot(on);
        const int c = __popcll(m);
        if (n + c > kInList) {
          flush(n);
          n = 0;
        }
        if (on) lst[n + lanes_below(m, lane)] = base + g * kWave + lane;
        n += c;
        cnt += c;
      }
    }
  }
  if (n > 0) flush(n);
  float* o = a.Iin + ((size_t)t * a.B + b) * (a.qn * kFwdThreads) + p0;
#pragma unroll
  for (int e = 0; e < PW; e += 4) *(f32x4*)(o + e) = f32x4{acc[e], acc[e + 1], acc[e + 2], acc[e + 3]};
  if (sl == 0 && lane == 0) a.nin[(size_t)t * a.B + b] = cnt;
}

// The first layer's input rows: their filter zbar over the block's steps
// (zstart: its value at the block's start) and their p bits, the same
// recursion as the forward's filter rows.  One thread per four consecutive
// inputs and batch element (32-bit words of x when rows allow, else bytes),
// the inputs of a 16-step chunk loaded per round trip (32-bit offsets from
// the block's x); the four inputs' 16-bit words of a chunk are adjacent (one
// 8-byte store).
__global__ __launch_bounds__(256) void input_filter_kernel(InputArgs a) {
  const int g = blockIdx.x * 256 + threadIdx.x, b = blockIdx.y;   // inputs 4 g .. 4 g + 3
  const int i0 = 4 * g;
  if (i0 >= a.n_in) return;
  const int ni = min(4, a.n_in - i0);
  const bool words = (a.n_in & 3) == 0 && ((uintptr_t)a.x & 3) == 0;
  const uint32_t stride = (uint32_t)a.B * (uint32_t)a.n_in;   // bytes per step
  float z[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    z[k] = k < ni ? a.zbar[(size_t)b * a.n_pre + i0 + k] : 0.0f;
    if (k < ni) a.zstart[(size_t)b * a.ldi + i0 + k] = z[k];
  }
  for (int t0 = 0; t0 < a.steps; t0 += kChunk) {
    uint32_t xv[kChunk];   // byte k: input i0 + k at step t0 + u
    uint32_t off = (uint32_t)t0 * stride + (uint32_t)b * a.n_in + i0;
#pragma unroll
    for (int u = 0; u < kChunk; ++u, off += stride) {
      xv[u] = 0;
      if (t0 + u < a.steps) {
        if (words) {
          xv[u] = *(const uint32_t*)(a.x + off);
        } else {
          for (int k = 0; k < ni; ++k) xv[u] |= (uint32_t)a.x[off + k] << (8 * k);
        }
      }
    }
    uint32_t m[4] = {0u, 0u, 0u, 0u};   // the chunk's bits of each input
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      if (t0 + u < a.steps) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const bool on = ((xv[u] >> (8 * k)) & 0xFFu) != 0;
          m[k] |= (on ? 1u : 0u) << u;
          z[k] = a.alpha * z[k] + (on ? 1.0f : 0.0f);
        }
      }
    }
    uint16_t* d = a.pbits + ((size_t)b * kKC + t0 / kChunk) * a.ldi + i0;
    if (ni == 4) {
      __builtin_nontemporal_store((unsigned long long)m[0] | ((unsigned long long)m[1] << 16) |
                                      ((unsigned long long)m[2] << 32) | ((unsigned long long)m[3] << 48),
                                  (unsigned long long*)d);
    } else {
      for (int k = 0; k < ni; ++k) __builtin_nontemporal_store((uint16_t)m[k], d + k);
    }
  }
#pragma unroll
  for (int k = 0; k < 4; ++k)
    if (k < ni) a.zbar[(size_t)b * a.n_pre + i0 + k] = z[k];
}

// ---------------------------------------------------------------- MFMA GEMM
// v_mfma_f32_16x16x4f32 operand layout (64 lanes, lane = r + 16*g):
//   A[16 x 4]:  lane holds A[r][g];  B[4 x 16]: lane holds B[g][r];
//   D[16 x 16]: lane holds D[4*g + q][r] in accumulator register q.
// Each lane takes its row's (NT) or column's (TN) values at 4 consecutive k
// of A and of Bm and feeds them to 4 MFMAs; both operands use the same k
// permutation, so the 4 MFMAs together contract 16 consecutive k.  One wave
// computes a 32x32 tile (2x2 blocks of 16x16); a block of 4 waves covers
// 32 (m) x 128 (n); blockIdx.z is the split of k.
__global__ __launch_bounds__(256) void gemm_nt_kernel(GemmArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int m0 = blockIdx.y * 32;
  const int n0 = (blockIdx.x * 4 + wave) * 32;
  if (n0 >= a.N) return;   // whole wave leaves; no block barrier in this kernel
  const int split = blockIdx.z;
  const int kb = split * a.k_chunk;
  const int ke = min(a.K, kb + a.k_chunk);
  const int r = lane & 15, g = lane >> 4;

  const float* pa0 = a.A + (size_t)(m0 + r) * a.lda + 4 * g;
  const float* pa1 = pa0 + (size_t)16 * a.lda;
  const float* pb0 = a.Bm + (size_t)(n0 + r) * a.ldb + 4 * g;
  const float* pb1 = pb0 + (size_t)16 * a.ldb;

  f32x4 c00 = {0.f, 0.f, 0.f, 0.f}, c01 = c00, c10 = c00, c11 = c00;
  for (int k = kb; k < ke; k += 16) {
    const f32x4 va0 = *(const f32x4*)(pa0 + k);
    const f32x4 va1 = *(const f32x4*)(pa1 + k);
    const f32x4 vb0 = *(const f32x4*)(pb0 + k);
    const f32x4 vb1 = *(const f32x4*)(pb1 + k);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      c00 = __builtin_amdgcn_mfma_f32_16x16x4f32(va0[q], vb0[q], c00, 0, 0, 0);
      c01 = __builtin_amdgcn_mfma_f32_16x16x4f32(va0[q], vb1[q], c01, 0, 0, 0);
      c10 = __builtin_amdgcn_mfma_f32_16x16x4f32(va1[q], vb0[q], c10, 0, 0, 0);
      c11 = __builtin_amdgcn_mfma_f32_16x16x4f32(va1[q], vb1[q], c11, 0, 0, 0);
    }
  }
  float* out = a.C + (size_t)split * a.split_stride;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int mA = m0 + 4 * g + q, mB = mA + 16;
    const int nA = n0 + r, nB = nA + 16;
    if (mA < a.M) {
      if (nA < a.N) out[(size_t)mA * a.ldc + nA] = c00[q];
      if (nB < a.N) out[(size_t)mA * a.ldc + nB] = c01[q];
    }
    if (mB < a.M) {
      if (nA < a.N) out[(size_t)mB * a.ldc + nA] = c10[q];
      if (nB < a.N) out[(size_t)mB * a.ldc + nB] = c11[q];
    }
  }
}

// Both operands stored k-major: lane (r, g) takes A[k][m] and Bm[k][n0 + r]
// for its four k of every 16-k chunk.  A wave covers 16*MB rows of m (all of
// them, M <= 16*MB) and 32 columns of n, so the large operand Bm is read once.
template <int MB>
__global__ __launch_bounds__(256) void gemm_tn_kernel(GemmArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int n0 = (blockIdx.x * 4 + wave) * 32;
  if (n0 >= a.N) return;
  const int split = blockIdx.z;
  const int kb = split * a.k_chunk;
  const int ke = min(a.K, kb + a.k_chunk);
  const int r = lane & 15, g = lane >> 4;
  f32x4 c[MB][2];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) c[mb][0] = c[mb][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 2
  for (int k = kb; k < ke; k += 16) {
    f32x4 va[MB], vb0, vb1;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const size_t kk = (size_t)(k + 4 * g + q);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) va[mb][q] = a.A[kk * a.lda + 16 * mb + r];
      vb0[q] = a.Bm[kk * a.ldb + n0 + r];
      vb1[q] = a.Bm[kk * a.ldb + n0 + 16 + r];
    }
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        c[mb][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(va[mb][q], vb0[q], c[mb][0], 0, 0, 0);
        c[mb][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(va[mb][q], vb1[q], c[mb][1], 0, 0, 0);
      }
  }
  float* out = a.C + (size_t)split * a.split_stride;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int m = 16 * mb + 4 * g + q;
      const int nA = n0 + r, nB = nA + 16;
      if (m < a.M) {
        if (nA < a.N) out[(size_t)m * a.ldc + nA] = c[mb][0][q];
        if (nB < a.N) out[(size_t)m * a.ldc + nB] = c[mb][1][q];
      }
    }
}

// Split-K partials added into an fp64 accumulator in split order.
__global__ __launch_bounds__(256) void accumulate_kernel(const float* part, int splits, size_t ss,
                                                        int M, int N, double* acc, int ld, int first) {
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)M * N) return;
  const int m = (int)(idx / N), n = (int)(idx % N);
  double s = first ? 0.0 : acc[(size_t)m * ld + n];
#pragma unroll 8
  for (int sp = 0; sp < splits; ++sp) s += (double)part[sp * ss + (size_t)m * N + n];
  acc[(size_t)m * ld + n] = s;
}

// ---------------------------------------------------------------- eligibility
// Over a block of K steps the recursion of one synapse (i, j) of batch
// element b,
//   e = psi_j (zbar_i - beta_j epsa);  ebar = kappa ebar + e;  g += L_j ebar;
//   epsa = psi_j zbar_i + (rho - beta_j psi_j) epsa,
// is linear in the block's starting traces E0 = ebar, A0 = epsa and in the
// presynaptic values zbar_{i,s}, with coefficients that depend only on
// (b, j, s).  So
//   ebar_K = kappa^K E0 + P_j A0 + sum_s zbar_{i,s} U_{j,s}
//   epsa_K = D_j A0           + sum_s zbar_{i,s} V_{j,s}
//   g     += c_j E0 + q_j A0  + sum_s zbar_{i,s} H_{j,s}
// Coefficients (d_s = rho - beta_j psi_s, M_s = sum_{t>=s} kappa^{t-s} L_t,
// N_s = sum_{r>s} beta_j psi_r M_r prod_{s<u<r} d_u):
//   H_s = psi_s (M_s - N_s),  c = kappa M_0,  q = -N_{-1},
//   U_s, P: the same with L replaced by the unit vector at the block's last
//   step,  V_s = psi_s prod_{u>s} d_u,  D = prod_u d_u.
// For LIF neurons beta_j = 0: N = 0, the epsa terms vanish.
// The filter is zbar_s = alpha^{s+1} Z + sum_{r<=s} alpha^{s-r} p_r (Z: its
// value at the block's start, p: the binary presynaptic values), so each sum
// is one over the binary p against the alpha-filtered coefficients
//   X'_r = sum_{s>=r} alpha^{s-r} X_s = X_r + alpha X'_{r+1},
// plus Z alpha X'_0.  p is exact in fp16, so each contraction takes one MFMA
// pass.  Written: U', H', V' as scaled pairs, and S [8][B][ldc]:
//   0 c  1 q  2 P  3 D  4 the scale exponents of U', H', V' (one byte each,
//   biased by 128, in the bits of the float)  5 alpha U'_0  6 alpha H'_0
//   7 alpha V'_0
// The sums over s are dense contractions (MFMA); the rest is elementwise.
// Two passes of the backward recursion: the first finds each array's largest
// magnitude (its scale), the second writes the scaled pairs chunk by chunk.
struct CoefState {
  float M = 0.0f, Mu = 0.0f, nx = 0.0f, nxu = 0.0f, Dsuf = 1.0f;   // backward recursion
  float up = 0.0f, hp = 0.0f, vp = 0.0f;                          // alpha-filtered U, H, V
  // step s (of `steps`); returns U'_s, H'_s, V'_s
  __device__ __forceinline__ void step(const CoefArgs& a, int s, float ps, float L, float bt,
                                       float& u, float& h, float& v) {
    const float d = a.rho - bt * ps;
    M = fmaf(a.kappa, M, L);
    Mu = (s == a.steps - 1) ? 1.0f : a.kappa * Mu;
    up = fmaf(a.alpha, up, ps * (Mu - nxu));
    hp = fmaf(a.alpha, hp, ps * (M - nx));
    vp = fmaf(a.alpha, vp, ps * Dsuf);
    nx = fmaf(bt * ps, M, d * nx);
    nxu = fmaf(bt * ps, Mu, d * nxu);
    Dsuf = d * Dsuf;
    u = up;
    h = hp;
    v = vp;
  }
};

__global__ __launch_bounds__(256) void coef_kernel(CoefArgs a) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const int b = blockIdx.y;
  if (j >= a.n_post) return;
  const float bt = (j < a.n_adaptive) ? a.beta : 0.0f;
  const int jt = j / kTileJ;
  const bool wv = jt < a.ol.n_jt_a;   // a tile holding adaptive neurons: V' too
  const float* __restrict__ psiK = a.psiK;
  const float* __restrict__ LK = a.LK;
  auto load_chunk = [&](int c, float (&ps)[kChunk], float (&L)[kChunk]) {
#pragma unroll
    for (int e = 0; e < kChunk; ++e) {
      const int s = kChunk * c + e;
      ps[e] = 0.0f;
      L[e] = 0.0f;
      if (s < a.steps) {
        const size_t row = ((size_t)s * a.Bp + b) * a.ldv + j;
        ps[e] = psiK[row];
        L[e] = LK[row];
      }
    }
  };
  float mU = 0.0f, mH = 0.0f, mV = 0.0f;
  {
    CoefState st;
    for (int c = a.kpad / kChunk - 1; c >= 0; --c) {
      float ps[kChunk], L[kChunk];
      load_chunk(c, ps, L);
#pragma unroll
      for (int e = kChunk - 1; e >= 0; --e) {
        const int s = kChunk * c + e;
        if (s >= a.steps) continue;
        float u, h, v;
        st.step(a, s, ps[e], L[e], bt, u, h, v);
        mU = fmaxf(mU, fabsf(u));
        mH = fmaxf(mH, fabsf(h));
        mV = fmaxf(mV, fabsf(v));
      }
    }
  }
  const int eU = pair_exponent(mU), eH = pair_exponent(mH), eV = pair_exponent(mV);
  const float sU = ldexpf(1.0f, eU), sH = ldexpf(1.0f, eH), sV = ldexpf(1.0f, eV);
  const size_t rs = (size_t)a.ol.cw;                // words between chunks
  uint32_t* o = a.O + (size_t)b * kKC * a.ol.cw + a.ol.tile(jt) + (j % kTileJ) * kChunk;
  CoefState st;
  for (int c = a.kpad / kChunk - 1; c >= 0; --c) {
    float ps[kChunk], L[kChunk];
    load_chunk(c, ps, L);
    float u[kChunk], v[kChunk], h[kChunk];
#pragma unroll
    for (int e = kChunk - 1; e >= 0; --e) {
      const int s = kChunk * c + e;
      if (s >= a.steps) {
        u[e] = v[e] = h[e] = 0.0f;
        continue;
      }
      st.step(a, s, ps[e], L[e], bt, u[e], h[e], v[e]);
    }
    // the tile's operands U, H (, V) one after the other, 1 KiB each
    store_pairs(o + c * rs, u, sU);
    store_pairs(o + c * rs + 256, h, sH);
    if (wv) store_pairs(o + c * rs + 512, v, sV);
  }
  const size_t so = (size_t)b * a.ldc + j, plane = (size_t)a.B * a.ldc;
  const uint32_t ex = (uint32_t)(eU + 128) | ((uint32_t)(eH + 128) << 8) | ((uint32_t)(eV + 128) << 16);
  const float out[8] = {a.kappa * st.M, -st.nx, -st.nxu, st.Dsuf, __uint_as_float(ex),
                        a.alpha * st.up, a.alpha * st.hp, a.alpha * st.vp};
#pragma unroll
  for (int k = 0; k < 8; ++k) a.S[k * plane + so] = out[k];
}

// Reset path kept in the gradient.  The membrane eligibility is then a
// per-synapse state V whose input is the binary presynaptic value p_{i,s};
// per step (v = V + p_s)
//   e = psi_j (v - beta_j A);  E = kappa E + e;  g += L_j E;
//   A = e + rho A;  V = alpha v - thr e,
// the same recursion as psi v + (rho - beta psi) A and
// (alpha - thr psi) v + thr beta psi A.  Over a block every output Y of
// E_K, g, A_K, V_K is linear in the block-start (V0, A0, E0) and in the p_s.
// The adjoint (lV, lA, lE) of Y with respect to the state before step s runs
// backwards from the unit vector of Y (zero for g):
//   tE = lE + [Y = g] L_s;  w = psi_s (lA + tE - thr lV);
//   lV = alpha lV + w;  lA = rho lA - beta w;  lE = kappa tE.
// p_s enters where V does, so Y's coefficient of p_s is lV after the update
// at step s, and the block-start state enters with (lV, lA, lE) at s = 0.
// Rows written: U = C_E, H = C_g, V = C_A (tiles holding adaptive neurons),
// W = C_V, as scaled pairs like coef_kernel's; S holds 16 planes:
//   0 gE  1 gA  2 gV  3 eA  4 eV  5 aA  6 aV  7 vA  8 vV
//   9 1/sU  10 1/sH  11 1/sV  12 1/sW  (E0 reaches E_K as kappa^K only and
//   reaches neither A_K nor V_K).
struct Adjoint {
  float v = 0.0f, a = 0.0f, e = 0.0f;
  __device__ __forceinline__ void step(const CoefArgs& A, float ps, float Lg, float bt) {
    const float te = e + Lg;
    const float w = ps * (a + te - A.thr * v);
    v = fmaf(A.alpha, v, w);
    a = fmaf(A.rho, a, -bt * w);
    e = A.kappa * te;
  }
  __device__ __forceinline__ float coef(const CoefArgs&) const { return v; }
};

// The same adjoint for any neuron step that is linear in its two state
// components (coefficients derived on the host): with the stored state
// sigma = H_I eps before the next input, per step
//   eps = sigma + b p;  e = psi (c . eps);  E = kappa E + e;  g += L E;
//   sigma' = A eps + r e,
// the adjoint of an output runs backwards as
//   tE = lE + [Y = g] L;  le = tE + r . l;  w = psi le;
//   l' = A^T l + c w;  lE = kappa tE,
// and p's coefficient is b . l' (v: component 0, a: component 1).  With
// A = diag(alpha, rho), b = (1, 0), r = (-thr, 1), c = (1, -beta) it is the
// reset-kept LIF/ALIF recursion above.
struct GenAdjoint {
  float v = 0.0f, a = 0.0f, e = 0.0f;
  __device__ __forceinline__ void step(const CoefArgs& A, float ps, float Lg, float) {
    const float te = e + Lg;
    const float le = fmaf(A.gr[1], a, fmaf(A.gr[0], v, te));
    const float w = ps * le;
    const float nv = fmaf(A.gc[0], w, fmaf(A.gA[1][0], a, A.gA[0][0] * v));
    const float na = fmaf(A.gc[1], w, fmaf(A.gA[1][1], a, A.gA[0][1] * v));
    v = nv;
    a = na;
    e = A.kappa * te;
  }
  __device__ __forceinline__ float coef(const CoefArgs& A) const { return fmaf(A.gb[1], a, A.gb[0] * v); }
};

template <typename Adj>
__global__ __launch_bounds__(256) void coef_rt_kernel(CoefArgs a) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const int b = blockIdx.y;
  if (j >= a.n_post) return;
  const float bt = (j < a.n_adaptive) ? a.beta : 0.0f;
  const int jt = j / kTileJ;
  const bool wv = jt < a.ol.n_jt_a;   // a tile holding adaptive neurons: V' too
  const float* __restrict__ psiK = a.psiK;
  const float* __restrict__ LK = a.LK;
  auto load_chunk = [&](int c, float (&ps)[kChunk], float (&L)[kChunk]) {
#pragma unroll
    for (int e = 0; e < kChunk; ++e) {
      const int s = kChunk * c + e;
      ps[e] = 0.0f;
      L[e] = 0.0f;
      if (s < a.steps) {
        const size_t row = ((size_t)s * a.Bp + b) * a.ldv + j;
        ps[e] = psiK[row];
        L[e] = LK[row];
      }
    }
  };
  // terminal adjoints: E_K, g, A_K, V_K
  auto init = [](Adj (&y)[4]) {
    y[0] = Adj{};
    y[0].e = 1.0f;
    y[1] = Adj{};
    y[2] = Adj{};
    y[2].a = 1.0f;
    y[3] = Adj{};
    y[3].v = 1.0f;
  };
  float mx[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  {
    Adj y[4];
    init(y);
    for (int c = a.kpad / kChunk - 1; c >= 0; --c) {
      float ps[kChunk], L[kChunk];
      load_chunk(c, ps, L);
#pragma unroll
      for (int e = kChunk - 1; e >= 0; --e) {
        if (kChunk * c + e >= a.steps) continue;
#pragma unroll
        for (int o = 0; o < 4; ++o) {
          y[o].step(a, ps[e], o == 1 ? L[e] : 0.0f, bt);
          mx[o] = fmaxf(mx[o], fabsf(y[o].coef(a)));
        }
      }
    }
  }
  float sc[4];
#pragma unroll
  for (int o = 0; o < 4; ++o) sc[o] = ldexpf(1.0f, pair_exponent(mx[o]));
  const size_t rs = (size_t)a.ol.cw;                // words between chunks
  uint32_t* o = a.O + (size_t)b * kKC * a.ol.cw + a.ol.tile(jt) + (j % kTileJ) * kChunk;
  Adj y[4];
  init(y);
  for (int c = a.kpad / kChunk - 1; c >= 0; --c) {
    float ps[kChunk], L[kChunk];
    load_chunk(c, ps, L);
    float x[4][kChunk];
#pragma unroll
    for (int e = kChunk - 1; e >= 0; --e) {
      const bool live = kChunk * c + e < a.steps;
#pragma unroll
      for (int o = 0; o < 4; ++o) {
        if (live) y[o].step(a, ps[e], o == 1 ? L[e] : 0.0f, bt);
        x[o][e] = live ? y[o].coef(a) : 0.0f;
      }
    }
    // the tile's operands U, H (, V), W one after the other, 1 KiB each
    store_pairs(o + c * rs, x[0], sc[0]);
    store_pairs(o + c * rs + 256, x[1], sc[1]);
    if (wv) store_pairs(o + c * rs + 512, x[2], sc[2]);
    store_pairs(o + c * rs + (wv ? 768 : 512), x[3], sc[3]);
  }
  const size_t so = (size_t)b * a.ldc + j, plane = (size_t)a.B * a.ldc;
  const float s16[13] = {y[1].e, y[1].a, y[1].v, y[0].a, y[0].v, y[2].a, y[2].v, y[3].a, y[3].v,
                         1.0f / sc[0], 1.0f / sc[1], 1.0f / sc[2], 1.0f / sc[3]};
#pragma unroll
  for (int k = 0; k < 13; ++k) a.S[k * plane + so] = s16[k];
}

// A workgroup of 4 waves owns a 256 (i) x 16 (j) tile of synapses and one
// split of the batch; wave w computes the 64 x 16 sub-tile of rows
// 64 w .. 64 w + 63.  Tall tiles let one shared-memory copy of a chunk of
// coefficient rows (which depend on j) serve 256 presynaptic rows, and all
// four waves read the same coefficient operand.
// For each batch element b of the split:
//  * MFMA contractions C_U, C_V, C_H = coef_b[j][s] x p_b[i][s] over the
//    block's steps (v_mfma_f32_16x16x32_f16 on the scaled fp16 pairs, four
//    16x16 blocks per wave stacked along i), 16 steps ("a chunk") at a time
//    and two chunks per wait and barrier ("a pair"), operands read from
//    shared memory;
//  * then the elementwise update of the traces, each read once and written
//    once (1 KiB contiguous per wave instruction), and of the gradient, at
//    the end of the element's own iteration.
// Operands stream through a ring of kRing pair slots in shared memory: the
// p bits of the tile's 256 rows (512 bytes per chunk; a wave copies its own
// 64 rows) and the tile's coefficient operands U, H (and V, W), one
// contiguous run per chunk in the tile-major layout (one operand of 1 KiB
// per copying wave), are copied by direct buffer-to-LDS loads (16 bytes per
// lane, no registers, the chunk's position in a scalar offset) up to
// kRing - 1 pairs ahead of the pair being contracted, across batch elements.
// An element's scalars (shared memory, double-buffered; with the block-start
// filter of the tile's rows) travel with its first pair; its block-start
// traces (registers) are loaded during its iteration, one 16x16 block per
// pair over its first four pairs.
// Waits: the copies of a wave complete in order, so a pair's copies are
// waited for with an exact vmcnt.  The workgroup barrier carries no memory
// fence (a fence would drain every copy in flight); shared-memory hazards are
// ordered by the waits and the barrier alone.
// Lane (r, g) of block bi holds the 4 columns j = j0 + 4 g ..+3 of row
// i = i0 + 64 w + 16 bi + r; the traces of a wave sub-tile are stored in
// exactly this order (block bi at bi KiB, lane l at 16 l bytes).  A wave whose
// 64 rows are all padding (past n_pre) reads and writes no traces.  The
// gradient of the batch elements of one launch is summed in fp32 per lane and
// added to the split's fp64 accumulator at the end.
// Workgroup order (trace_kernel): the row tiles of one column tile and batch
// split, which share every coefficient chunk, run on one XCD.
// Buffer access: a wave-uniform base with a byte range (accesses outside it
// read zero and write nothing) and a 32-bit per-lane byte offset.  The trace
// streams use the non-temporal cache policy (bit 1 of the policy operand):
// each trace is touched once per block, and keeping it out of the caches
// leaves room for the operand tiles that neighbouring workgroups reuse.
constexpr int kNonTemporal = 2;
__device__ __forceinline__ f32x4 bload(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNonTemporal));
}
__device__ __forceinline__ void bstore(__amdgpu_buffer_rsrc_t r, uint32_t off, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, off, 0, kNonTemporal);
}

constexpr int kRing = 4;                              // slots of two chunks
constexpr int kOpBytes = kTileJ * 64;                 // one coefficient operand of a chunk: 16 rows x 64 B
constexpr int kPBytes = kTileI * 2;                   // the chunk's p bits: 256 rows x 16 bits
constexpr int kWaveRows = kTileI / 4;                 // rows of a wave sub-tile
constexpr uint32_t kSubTileBytes = kWaveRows * kTileJ * 4;   // a wave's traces of one array (4 KiB)
constexpr int kScalWave = 256;                        // floats of one wave's scalar copy (64 lanes x 16 B)

// s_waitcnt immediate that waits for vmcnt <= n only (gfx9 encoding)
constexpr int vm_wait(int n) { return (n & 0xF) | ((n >> 4) << 14) | 0x70 | 0xF00; }

__device__ __forceinline__ void wg_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Calls f(std::integral_constant<int, I>) for I = 0, 1, ... in order.
template <typename F, int... I>
__device__ __forceinline__ void for_each_index(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}

typedef __attribute__((address_space(3))) void lds_void;
// Lane l copies 16 bytes at byte voff + soff of the buffer r to lds + 16 l
// (soff: a wave-uniform offset, so stepping through chunks costs no vector
// instructions).
__device__ __forceinline__ void dma16b(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, void* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)lds, 16, voff, soff, 0, 0);
}

// RT = false: the reset-stopped recursion (contractions U', H' and, for
// tiles holding adaptive neurons, V'; traces ebar, epsa; coef_kernel).  RT =
// true: the reset path kept (coef_rt_kernel): contractions U = C_E, H = C_g,
// W = C_V and V = C_A; traces ebar, epsv and epsa.  Either way the
// presynaptic operand is the binary p, exact in fp16, so each contraction
// takes one MFMA pass.
template <bool ALIF, int NCH, bool RT>
struct TraceTile {
  // The chunks of a batch element are taken two at a time ("pairs", 32
  // steps; the last pair of an odd chunk count holds one): one wait, one
  // barrier and one batch of shared-memory reads per pair.
  static constexpr int NS = (NCH + 1) / 2;                    // pairs per batch element
  static constexpr int in_pair(int s) { return 2 * s + 1 < NCH ? 2 : 1; }   // chunks of pair s
  static constexpr int RING = kRing;                          // pair slots
  static constexpr int PREF = RING - 1;                       // pairs copied ahead
  // half a slot: a chunk's p bits (256 rows x 16 bits), then the
  // coefficient operands U, H, V (and W) of 16 rows x 64 B each (V's place is
  // kept in tiles without adaptive neurons)
  static constexpr int NOPS = RT ? 4 : 3;
  static constexpr int HSLOT = kPBytes + NOPS * kOpBytes;     // bytes per chunk
  static constexpr int SLOT = 2 * HSLOT / 4;                  // floats per slot
  static constexpr int PLANES = RT ? kScalarPlanesRT : kScalarPlanes;
  static constexpr int PPW = PLANES / 4;                      // planes copied per wave
  // one scalar buffer: per wave kScalWave floats = its PPW planes of the 16
  // columns, then (reset-stopped form) the block-start filter of its 64 rows
  static constexpr int SCAL = 4 * kScalWave;
  static constexpr int ZOFF = 64;                             // filter offset in a wave's part
  static_assert(PPW * kTileJ <= ZOFF, "planes overlap the filter");
  static constexpr size_t SMEM = sizeof(float) * (RING * SLOT + 2 * SCAL);
  // pairs in flight ahead; fewer than NS so that a batch element's copies
  // never reach past the next element's first pair
  static constexpr int D = NS == 1 ? 1 : (NS - 1 < PREF ? NS - 1 : PREF);
  // Copies per wave per chunk: its p rows, and one coefficient operand for
  // the copying waves (wave X copies operand X: U, H, and V / W when present).
  static constexpr int SC = RT ? 1 : 2;                         // scalar copies per wave (planes, filter)
  static constexpr int EA = 4 * (1 + (ALIF ? 1 : 0) + (RT ? 1 : 0));   // trace loads per element
  static constexpr int ops(int s, bool cp) { return in_pair(s) * (1 + (cp ? 1 : 0)) + (s == 0 ? SC : 0); }
  // The block-start traces are loaded one 16 x 16 block bi of each trace per
  // pair over the element's first four pairs (all at pair 0 with fewer
  // pairs), after that pair's copies: spread out, the loads of a batch element
  // do not arrive at the memory system at once, and the copies issued after
  // them (which complete in order behind them) are not held up by a burst.
  static constexpr int NT = EA / 4;                              // traces per element
  static constexpr bool spread = NS >= 4;
  static constexpr int tl(int s) { return spread ? (s < 4 ? NT : 0) : (s == 0 ? EA : 0); }
  // Loads issued after those of pair s when it is waited for: the copies of
  // pairs s+1 .. s+D-1 (past the end of the batch element: the next
  // element's, if there is one), and the element's trace loads when they
  // were issued in between (at pair 0, after that pair's copies).  Loads
  // complete in order, so at most that many outstanding operations means
  // pair s has landed, whatever stores are still in flight.
  static constexpr int pending(int ps, bool next, bool cp) {
    int n = 0;
    for (int i = ps - D; i < ps; ++i) n += i >= 0 ? tl(i) : 0;
    for (int m = ps + 1; m <= ps + D - 1; ++m)
      n += m < NS ? ops(m, cp) : (next ? ops(m - NS, cp) : 0);
    return n;
  }
  static_assert(pending(1, true, true) <= 63, "vmcnt range");

  const TraceArgs& a;
  float* sm;
  int i0, j0, it, jt, split, lane, r, g, w;
  bool first, live, copier;
  uint32_t pvoff, cvoff;          // this lane's byte offsets in the p and coefficient copies
  const char* opbase;             // the coefficient operand this wave copies (copier waves)

  __device__ __forceinline__ TraceTile(const TraceArgs& a_, float* sm_, int it_, int jt_, int split_,
                                       bool first_)
      : a(a_), sm(sm_), i0(it_ * kTileI), j0(jt_ * kTileJ), it(it_), jt(jt_), split(split_),
        first(first_) {
    lane = threadIdx.x & 63;
    r = lane & 15;
    g = lane >> 4;
    w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave index, uniform
    live = i0 + kWaveRows * w < a.n_pre;                    // the wave holds a real row
    copier = (w < 2) || (w == 2 && ALIF) || (w == 3 && RT);
    // p: the bits of rows i0 + 64 w .. +63 are one contiguous 128-byte run;
    // coefficients: lane l takes row l / 4 of the 16 columns, 16-byte unit
    // (l % 4) ^ ((row / 2) % 4) (see issue)
    pvoff = (uint32_t)(i0 + kWaveRows * w) * 2u + (uint32_t)(lane & 7) * 16u;
    const int row = lane >> 2;
    cvoff = (uint32_t)row * 64u + (uint32_t)((lane & 3) ^ ((row >> 1) & 3)) * 16u;
    // operand w of the tile (U, H, V, W; W follows H where the tile has no V)
    opbase = (const char*)(a.O + a.ol.tile(jt_)) + (w == 3 && !ALIF ? 2 : w) * kOpBytes;
  }

  // The lane index computed where it is used, from an operand the compiler
  // cannot hoist: offsets derived from it then take no register across the
  // element loop (at the register cap such values were spilled, and each
  // reload waited for every copy in flight).
  __device__ __forceinline__ static uint32_t lane_here() {
    uint32_t ones = ~0u;
    asm volatile("" : "+s"(ones));
    return __builtin_amdgcn_mbcnt_hi(ones, __builtin_amdgcn_mbcnt_lo(ones, 0u));
  }

  __device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const float* base, int n_t, int b,
                                                             uint32_t bytes) const {
    const size_t t = ((size_t)b * (a.n_pre_pad / kTileI) + it) * n_t + jt;
    return make_rsrc((const char*)base + (t * 4 + w) * kSubTileBytes, live ? bytes : 0u);
  }

  // Copies of the NC chunks c, c + 1 (< NC) of batch element b into pair
  // slot sl: wave w copies the p bits of its 64 rows (one 16-bit word per
  // row and chunk, 128 bytes, lanes 0-7), and a copying wave its coefficient
  // operand of the tile (lane l: row l / 4, its 16-byte unit
  // u = (l % 4) ^ ((row / 2) % 4) stored at position l % 4, which keeps the
  // MFMA operand reads free of bank conflicts).  With chunk 0 also the
  // scalars (planes PPW w .. PPW w + PPW - 1 of the 16 columns, and the
  // block-start filter of the wave's rows) into scalar buffer par.  The
  // copies are issued in two parts (P = 0: p; P = 1: the coefficient operand
  // and the scalars), placed between MFMAs so that the vector-memory path
  // works while the matrix cores do; the order of all copies is that of the
  // full issue.
  template <int P, int NC>
  __device__ __forceinline__ void issue(int b_, int c, int sl, int par) const {
    const int b = __builtin_amdgcn_readfirstlane(b_);   // wave-uniform: scalar address arithmetic
    char* slot = (char*)(sm + sl * SLOT);
    if constexpr (P == 0) {
      const uint32_t estride = (uint32_t)(kKC * a.ldi * 2);          // bytes of one element
      const auto pr = make_rsrc((const char*)a.pbits + (size_t)b * estride, estride);
      // the chunk offsets computed here (kept out of scalar registers
      // across the loop)
      uint32_t cs = (uint32_t)(a.ldi * 2);
      asm volatile("" : "+s"(cs));
      // the wave's 64 rows: 128 bytes, lanes 0-7 (one instruction per wave
      // and chunk)
#pragma unroll
      for (int h = 0; h < NC; ++h)
        if (lane < 8) dma16b(pr, pvoff, (uint32_t)(c + h) * cs, slot + h * HSLOT + kWaveRows * w * 2);
    } else {
      if (copier) {
        const uint32_t estride = (uint32_t)(kKC * a.ol.cw * 4);      // bytes of one element
        const auto cr = make_rsrc(opbase + (size_t)b * estride, estride);
        uint32_t cs = (uint32_t)(a.ol.cw * 4);
        asm volatile("" : "+s"(cs));
#pragma unroll
        for (int h = 0; h < NC; ++h)
          dma16b(cr, cvoff, (uint32_t)(c + h) * cs, slot + h * HSLOT + kPBytes + w * kOpBytes);
      }
      if (c == 0) {
        float* sb = sm + RING * SLOT + par * SCAL + w * kScalWave;
        // lanes 0 .. 4 PPW - 1: plane PPW w + l / 4, columns 4 (l % 4) .. +3;
        // lanes 16-31 (reset-stopped form): the filter of rows 64 w + 4 (l - 16) .. +3.
        // Buffer loads from a per-element scalar base and 32-bit lane
        // offsets (computed here from the lane index).
        const uint32_t l = lane_here();
        const uint32_t pst = (uint32_t)(a.B * a.ldc) * 4u;           // bytes between planes
        const auto sr = make_rsrc(a.S + (size_t)b * a.ldc + j0, (uint32_t)(PLANES - 1) * pst + kTileJ * 4u);
        if (l < 4u * PPW) dma16b(sr, (uint32_t)(PPW * w + (l >> 2)) * pst + (l & 3u) * 16u, 0u, sb);
        if constexpr (!RT) {
          const auto zr = make_rsrc(a.zstart + (size_t)b * a.ldi + i0 + kWaveRows * w, kWaveRows * 4u);
          if (l >= 16u && l < 32u) dma16b(zr, (l - 16u) * 16u, 0u, sb);
        }
      }
    }
  }
  // all copies of pair PS (chunks 2 PS and 2 PS + 1 when there is one)
  template <int PS>
  __device__ __forceinline__ void issue_all(int b, std::integral_constant<int, PS>, int sl, int par) const {
    issue<0, in_pair(PS)>(b, 2 * PS, sl, par);
    issue<1, in_pair(PS)>(b, 2 * PS, sl, par);
  }

  // block-start traces of batch element b into E, A (and Vm).  In the first
  // block after a reset (and for a wave of padding rows) they are zero: the
  // loads then get an empty range, so they read zero without touching memory
  // and still count as issued loads (the waits above count them).
  // blocks x0 .. x1 - 1 of each
  __device__ __forceinline__ void load_traces(int b, int x0, int x1, f32x4 (&E)[4], f32x4 (&A)[4],
                                              f32x4 (&Vm)[4]) const {
    const uint32_t range = first ? 0u : kSubTileBytes;
    const auto eR = tile_rsrc(a.ebar, a.n_jt, b, range);
#pragma unroll
    for (int x = 0; x < 4; ++x)
      if (x >= x0 && x < x1) E[x] = bload(eR, x * 1024u + lane * 16u);
    if constexpr (ALIF) {
      const auto aR = tile_rsrc(a.epsa, a.n_jt_a, b, range);
#pragma unroll
      for (int x = 0; x < 4; ++x)
        if (x >= x0 && x < x1) A[x] = bload(aR, x * 1024u + lane * 16u);
    }
    if constexpr (RT) {
      const auto vR = tile_rsrc(a.epsv, a.n_jt, b, range);
#pragma unroll
      for (int x = 0; x < 4; ++x)
        if (x >= x0 && x < x1) Vm[x] = bload(vR, x * 1024u + lane * 16u);
    }
  }

  // traces and gradient of the k-th batch element from its contractions
  // (accumulated in the scaled units of the fp16 pairs)
  __device__ __forceinline__ void finish(int k, const f32x4 (&E)[4], const f32x4 (&A)[4],
                                         const f32x4 (&Vm)[4], const f32x4 (&cU)[4],
                                         const f32x4 (&cV)[4], const f32x4 (&cH)[4],
                                         const f32x4 (&cW)[4], f32x4 (&gacc)[4]) const {
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
    const int b = split + k * a.n_split;
    const float* st = sm + RING * SLOT + (k & 1) * SCAL;
    const auto eR = tile_rsrc(a.ebar, a.n_jt, b, kSubTileBytes);
    const auto aR = ALIF ? tile_rsrc(a.epsa, a.n_jt_a, b, kSubTileBytes) : eR;
    const auto vR = RT ? tile_rsrc(a.epsv, a.n_jt, b, kSubTileBytes) : eR;
    const int cj = 4 * (int)((lane_here() >> 4) & 3u);   // this lane group's columns
    auto plane = [&](int p) {
      return *(const f32x4*)(st + (p / PPW) * kScalWave + (p % PPW) * kTileJ + cj);
    };
    if constexpr (!RT) {
      // c, q, P, D, scale exponents, alpha U'_0, alpha H'_0, alpha V'_0
      // (coef_kernel); the block-start filter Z of row i after them.  One
      // output at a time, with the planes it needs, so that few registers
      // are live beside the contractions.
      // 2^-e from the biased exponent byte at bit `sh`
      auto inv_scale = [&](int sh) {
        const f32x4 ex = plane(4);
        f32x4 f;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          f[q] = __uint_as_float((uint32_t)(255 - (int)((__float_as_uint(ex[q]) >> sh) & 0xFF)) << 23);
        return f;
      };
      const float* zrow = st + w * kScalWave + ZOFF;
#pragma unroll
      for (int bi = 0; bi < 4; ++bi) {
        const f32x4 e0 = first ? zero : E[bi];
        const f32x4 a0 = (first || !ALIF) ? zero : A[bi];
        const float Z = zrow[16 * bi + r];
        const uint32_t o = bi * 1024u + lane * 16u;
        {
          const f32x4 P = ALIF ? plane(2) : zero, zU = plane(5), fU = inv_scale(0);
          f32x4 ek;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            ek[q] = fmaf(a.kappa_K, e0[q], fmaf(P[q], a0[q], fmaf(zU[q], Z, cU[bi][q] * fU[q])));
          bstore(eR, o, ek);
        }
        {
          const f32x4 c = plane(0), qq = plane(1), zH = plane(6), fH = inv_scale(8);
#pragma unroll
          for (int q = 0; q < 4; ++q)
            gacc[bi][q] += fmaf(c[q], e0[q], fmaf(qq[q], a0[q], fmaf(zH[q], Z, cH[bi][q] * fH[q])));
        }
        if constexpr (ALIF) {
          const f32x4 Dd = plane(3), zV = plane(7), fV = inv_scale(16);
          f32x4 ak;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            ak[q] = fmaf(Dd[q], a0[q], fmaf(zV[q], Z, cV[bi][q] * fV[q]));
          bstore(aR, o, ak);
        }
      }
    } else {
      // gE gA gV eA eV aA aV vA vV 1/sU 1/sH 1/sV 1/sW (coef_rt_kernel)
      const f32x4 gE = plane(0), gV = plane(2), eV = plane(4), vV = plane(8);
      const f32x4 gA = ALIF ? plane(1) : zero, eA = ALIF ? plane(3) : zero;
      const f32x4 aA = ALIF ? plane(5) : zero, aV = ALIF ? plane(6) : zero;
      const f32x4 vA = ALIF ? plane(7) : zero;
      const f32x4 fU = plane(9), fH = plane(10), fW = plane(12);
      const f32x4 fV = ALIF ? plane(11) : zero;
#pragma unroll
      for (int bi = 0; bi < 4; ++bi) {
        const f32x4 e0 = first ? zero : E[bi];
        const f32x4 v0 = first ? zero : Vm[bi];
        const f32x4 a0 = (first || !ALIF) ? zero : A[bi];
        f32x4 ek, ak, gk, vk;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          ek[q] = fmaf(a.kappa_K, e0[q], fmaf(eV[q], v0[q], fmaf(eA[q], a0[q], cU[bi][q] * fU[q])));
          gk[q] = fmaf(gE[q], e0[q], fmaf(gV[q], v0[q], fmaf(gA[q], a0[q], cH[bi][q] * fH[q])));
          vk[q] = fmaf(vV[q], v0[q], fmaf(vA[q], a0[q], cW[bi][q] * fW[q]));
          ak[q] = fmaf(aV[q], v0[q], fmaf(aA[q], a0[q], cV[bi][q] * fV[q]));
        }
        gacc[bi] += gk;
        const uint32_t o = bi * 1024u + lane * 16u;
        bstore(eR, o, ek);
        bstore(vR, o, vk);
        if constexpr (ALIF) bstore(aR, o, ak);
      }
    }
  }

  __device__ __forceinline__ void run() const {
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
    const int nk = (a.B - split + a.n_split - 1) / a.n_split;
    f32x4 gacc[4], cU[4], cV[4], cH[4], cW[4], E[4], A[4], Vm[4];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      gacc[x] = zero;
      cU[x] = cV[x] = cH[x] = cW[x] = zero;
      E[x] = A[x] = Vm[x] = zero;
    }
    for_each_index([&](auto pc) { issue_all(split, pc, decltype(pc)::value, 0); },
                   std::make_integer_sequence<int, D>{});
#pragma nounroll
    for (int k = 0; k < nk; ++k) {
      const int b = split + k * a.n_split;
      const bool next = k + 1 < nk;
      auto pair = [&](auto psc) {
        constexpr int ps = decltype(psc)::value;
        constexpr int NC = in_pair(ps);
        const int n = k * NS + ps;
        if (copier) {
          if (next)
            __builtin_amdgcn_s_waitcnt(vm_wait(pending(ps, true, true)));
          else
            __builtin_amdgcn_s_waitcnt(vm_wait(pending(ps, false, true)));
        } else {
          if (next)
            __builtin_amdgcn_s_waitcnt(vm_wait(pending(ps, true, false)));
          else
            __builtin_amdgcn_s_waitcnt(vm_wait(pending(ps, false, false)));
        }
        wg_barrier();   // pair n is in shared memory; slot (n - 1) % RING is free
        // copies of pair n + D (part P), placed inside the MFMA section
        constexpr int s2 = ps + D;
        auto issue_next = [&](auto pc) {
          constexpr int P = decltype(pc)::value;
          if constexpr (s2 < NS)
            issue<P, in_pair(s2 < NS ? s2 : 0)>(b, 2 * s2, (n + D) % RING, k & 1);
          else if (next)
            issue<P, in_pair(s2 - NS >= 0 ? s2 - NS : 0)>(b + a.n_split, 2 * (s2 - NS), (n + D) % RING,
                                                          (k + 1) & 1);
        };

        // Per output block and contraction X, one fp16 MFMA (K = 32) per
        // chunk of 16 steps.  Lane g holds the 8 k slots of steps 4g..4g+3:
        // A = X's unit as it is (the four hi halves, then the four lo
        // halves; row r of the 16 columns, the same for every wave), B = the
        // four p values twice, which sums X_hi p + X_lo p (p is the binary
        // presynaptic value, exact in fp16).
        const char* slot = (const char*)(sm + (n % RING) * SLOT);
        const int sw = (r >> 1) & 3;   // unit order of this lane's row
        const f16x8 zero8 = {};
        // Per output block and contraction X, two fp16 MFMAs (K = 32) per
        // pair of chunks: lane group g holds the 8 k slots of pair steps
        // 8g .. 8g+7 (chunk g / 2 of the pair), the first MFMA takes their hi
        // halves, the second their lo halves, each against the same 8 p
        // values, which sums X_hi p + X_lo p (p is the binary presynaptic
        // value, exact in fp16).  A pair of one chunk (the last of an odd
        // count) leaves lane groups 2 and 3 with zero operands.
        const bool none = NC == 1 && g >= 2;
        const char* hs = slot + (g >> 1) * HSLOT;   // this lane's chunk
        // the pair's shared-memory reads in one batch: the hi and lo units of
        // each coefficient operand and the p words of the four row blocks
        f16x8 axh[4], axl[4];
        uint32_t pw[4];
#pragma unroll
        for (int X = 0; X < 4; ++X) {
          const bool has = (X < 2) || (X == 2 && ALIF) || (X == 3 && RT);
          const char* row = hs + kPBytes + X * kOpBytes + r * 64;
          axh[X] = has ? *(const f16x8*)(row + (((g & 1) ^ sw) << 4)) : zero8;
          axl[X] = has ? *(const f16x8*)(row + (((2 + (g & 1)) ^ sw) << 4)) : zero8;
          if (NC == 1) {
            axh[X] = none ? zero8 : axh[X];
            axl[X] = none ? zero8 : axl[X];
          }
        }
#pragma unroll
        for (int bi = 0; bi < 4; ++bi)
          pw[bi] = *(const uint16_t*)(hs + (kWaveRows * w + 16 * bi + r) * 2);
        // pair steps 8g .. 8g+7 of row 16 bi + r of the wave: eight p bits n
        // -> the fp16 words (p0, p1), (p2, p3), (p4, p5), (p6, p7) (1.0 =
        // 0x3C00): with x = n (1 + 2^15), bits 2m and 2m + 16 of x are p_2m
        // and p_2m+1, so each word is one mask and one multiply (24-bit
        // operands); the 16 rows' words are 32 consecutive bytes, read by
        // every g alike
        auto expand = [&](int bi) {
          uint32_t x = __builtin_amdgcn_ubfe(pw[bi], 8 * (g & 1), 8) * 0x8001u;
          if (NC == 1) x = none ? 0u : x;
          return __builtin_bit_cast(f16x8, u32x4{(x & 0x10001u) * 0x3C00u, (x & 0x40004u) * 0xF00u,
                                                  (x & 0x100010u) * 0x3C0u, (x & 0x400040u) * 0xF0u});
        };
        auto mfma = [&](const f16x8 (&ax)[4], const f16x8& bz, int bi) {
          cU[bi] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ax[0], bz, cU[bi], 0, 0, 0);
          cH[bi] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ax[1], bz, cH[bi], 0, 0, 0);
          if constexpr (ALIF)
            cV[bi] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ax[2], bz, cV[bi], 0, 0, 0);
          if constexpr (RT)
            cW[bi] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ax[3], bz, cW[bi], 0, 0, 0);
        };
        // the pair's MFMAs at a raised issue priority: a wave whose operands
        // have arrived keeps the matrix pipe busy ahead of the waves still
        // reading theirs (still below the forward's)
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(1);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int b2 = 0; b2 < 4; b2 += 2) {
          // two row blocks at a time: their hi MFMAs, then their lo MFMAs,
          // so that an accumulator's two MFMAs are not back to back
          const f16x8 bz0 = expand(b2), bz1 = expand(b2 + 1);
          mfma(axh, bz0, b2);
          mfma(axh, bz1, b2 + 1);
          if (b2 == 0) {
            __builtin_amdgcn_sched_barrier(0);
            issue_next(std::integral_constant<int, 0>{});
            __builtin_amdgcn_sched_barrier(0);
          }
          mfma(axl, bz0, b2);
          mfma(axl, bz1, b2 + 1);
          if (b2 == 0) {
            __builtin_amdgcn_sched_barrier(0);
            issue_next(std::integral_constant<int, 1>{});
            // the element's block-start traces, after pair 0's copies
            if constexpr (spread && ps < 4)
              load_traces(b, ps, ps + 1, E, A, Vm);
            else if constexpr (!spread && ps == 0)
              load_traces(b, 0, 4, E, A, Vm);
            __builtin_amdgcn_sched_barrier(0);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(0);
        __builtin_amdgcn_sched_barrier(0);
      };
      for_each_index(pair, std::make_integer_sequence<int, NS>{});
      // The element's traces and gradient.  Its block-start traces were
      // loaded in this iteration (at pair 0), so the compiler's wait for them
      // counts only the loads issued since (no drain of the copies in flight
      // ahead); its scalars arrived with pair 0.  The scalar buffer of this
      // element's parity is next written with the copies of element k + 2's
      // first pair, after at least one more barrier.
      finish(k, E, A, Vm, cU, cV, cH, cW, gacc);
#pragma unroll
      for (int x = 0; x < 4; ++x) cU[x] = cV[x] = cH[x] = cW[x] = zero;
    }
    // the split's fp64 accumulator (row-major [n_pre_pad][ldj]); rows past
    // n_pre and columns past n_post are not written
    const int jb = j0 + 4 * (int)((lane_here() >> 4) & 3u);
    if (!live || jb >= a.n_post) return;
    double* accp = a.acc + (size_t)split * a.acc_stride;
#pragma unroll
    for (int bi = 0; bi < 4; ++bi) {
      const int i = i0 + kWaveRows * w + 16 * bi + r;
      if (i >= a.n_pre) continue;
      double* p = accp + (size_t)i * a.ldj + jb;
#pragma unroll
      for (int q = 0; q < 4; ++q) p[q] = (first ? 0.0 : p[q]) + (double)gacc[bi][q];
    }
  }
};

// Workgroup order: a group is one column tile jt of one batch split; its row
// tiles (which read the same coefficient chunks of the same batch elements)
// are consecutive workgroups of one XCD.  Workgroups go round-robin over the
// eight XCDs, so workgroup L belongs to XCD L % 8 and is the (L / 8)-th of
// that XCD; group G = 8 g + x is the g-th group of XCD x.  Dispatched one
// after the other on one XCD, the row tiles of a group start together and,
// being of one kind (a tile holding any adaptive neuron takes the path with
// the adaptation trace), advance together, so each coefficient chunk is
// fetched into that XCD's L2 once for all of them.  Workgroups past the last
// group exit at once.  One kernel per chunk count NCH = kpad / 16 (the host
// picks it), so that each holds only its own two variants.
// Three workgroups per compute unit for the reset-stopped form (its
// variants fit 168 registers), two with the reset path kept.
template <bool RT, int NCH>
__global__ __launch_bounds__(256, RT ? 2 : 3) void trace_kernel(TraceArgs a) {
  extern __shared__ __attribute__((aligned(16))) float trace_smem[];
  const int n_it = a.n_pre_pad / kTileI;
  const int L = blockIdx.x, x = L & 7, pos = L >> 3;
  const int gl = pos / n_it, it = pos - gl * n_it;
  const int G = gl * 8 + x;
  if (G >= a.n_jt * a.n_split) return;
  const int split = G / a.n_jt, jt = G - split * a.n_jt;
  const bool first = a.first != 0;
  if (jt < a.n_jt_a)
    TraceTile<true, NCH, RT>(a, trace_smem, it, jt, split, first).run();
  else
    TraceTile<false, NCH, RT>(a, trace_smem, it, jt, split, first).run();
}
// shared memory of the two variants (the same for every chunk count)
constexpr size_t kTraceSmemOf(bool rt) {
  return rt ? TraceTile<true, 16, true>::SMEM : TraceTile<true, 16, false>::SMEM;
}

// ---------------------------------------------------------------- gradient read-out
// 32x32 tiles through shared memory: acc is [i][j], dW is [j][i].
// The read-out of a call to eprop_get_grads in one launch; blockIdx.z picks
// the job: 2 l, layer l's dW (32 x 32 tiles on x, y, transposed through
// shared memory, the split accumulators summed in split order); 2 l + 1,
// layer l's dW_out (y = 0 only, one element per thread along x); 2 L, the
// loss (one thread, a fixed summation order over layers and batch elements).
__global__ __launch_bounds__(256) void readout_kernel(ReadoutArgs r) {
  const int job = blockIdx.z;
  if (job == 2 * r.n_layers) {
    if (threadIdx.x != 0 || blockIdx.x != 0 || blockIdx.y != 0) return;
    double s = 0.0;
    for (int l = 0; l < r.n_layers; ++l)
      for (int b = 0; b < r.B; ++b) s += r.lossacc[(size_t)l * r.layer_stride + b];
    *r.loss = s;
    return;
  }
  const GradsArgs& a = r.g[job >> 1];
  if (job & 1) {
    if (blockIdx.y != 0) return;
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (long long)a.K * a.n_post) return;
    const int k = (int)(idx / a.n_post), j = (int)(idx % a.n_post);
    a.dWout[(size_t)k * a.n_post + j] = a.valid ? (float)a.accout[(size_t)k * a.ld_acc + j] : 0.0f;
    return;
  }
  // the whole workgroup leaves together (its tile lies past the matrix)
  if ((int)blockIdx.x * 32 >= a.n_pre || (int)blockIdx.y * 32 >= a.n_post) return;
  __shared__ double tile[32][33];
  const int i0 = blockIdx.x * 32, j0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;   // 32 x 8
  for (int yy = ty; yy < 32; yy += 8) {
    const int i = i0 + yy, j = j0 + tx;
    double v = 0.0;
    if (a.valid && i < a.n_pre && j < a.n_post)
      for (int sp = 0; sp < a.n_split; ++sp) v += a.acc[sp * a.acc_stride + (size_t)i * a.ldj + j];
    tile[yy][tx] = v;
  }
  __syncthreads();
  for (int yy = ty; yy < 32; yy += 8) {
    const int j = j0 + yy, i = i0 + tx;
    if (j < a.n_post && i < a.n_pre) {
      const bool diag = a.recurrent && i == a.n_inl + j;
      a.dW[(size_t)j * a.n_pre + i] = diag ? 0.0f : (float)tile[tx][yy];
    }
  }
}

// Workgroups of the weight-packing kernels: a fixed grid walks the weights,
// so that the largest |k| takes one global atomic per workgroup.
constexpr int kPackBlocks = 1024;

// The largest |k| of a workgroup's exact weights (kmax: the thread's) into
// ok[1]: a maximum in shared memory, then one global atomic per workgroup
// (the result does not depend on the order).
__device__ __forceinline__ void max_k(int* ok, int kmax) {
  __shared__ int smax;
  if (threadIdx.x == 0) smax = 0;
  __syncthreads();
  if (kmax > 0) atomicMax(&smax, kmax);
  __syncthreads();
  if (threadIdx.x == 0 && smax > 0) atomicMax(ok + 1, smax);
}

__global__ __launch_bounds__(256) void pack16_kernel(const float* W, int n_rec, int n_pre,
                                                     int16_t* W16, int qn, int* ok) {
  const long long n = (long long)n_rec * n_pre;
  int kmax = 0;
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < n;
       idx += (long long)gridDim.x * blockDim.x) {
    const float k = W[idx] * 16384.0f;
    const bool exact = k == rintf(k) && fabsf(k) <= 32767.0f;
    if (!exact) ok[0] = 0;   // every thread that finds one writes the same value
    else kmax = max(kmax, (int)fabsf(k));
    const int j = (int)(idx / n_pre), i = (int)(idx % n_pre);
    W16[(size_t)i * (qn * kFwdThreads) + fwd_position(j, qn)] =
        exact ? (int16_t)k : (int16_t)0;
  }
  max_k(ok, kmax);
}

// Weights on the 2^-14 grid: rint(x 2^14) 2^-14 in fp64 (ties to even).
__device__ __forceinline__ float on_grid(double x) { return (float)(rint(x * 16384.0) / 16384.0); }

// One thread per (i, j), j fastest (coalesced over the accumulators and Wt).
__global__ __launch_bounds__(256) void online_w_kernel(OnlineArgs a) {
  const long long n = (long long)a.n_rec * a.n_pre;
  int kmax = 0;
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < n;
       idx += (long long)gridDim.x * blockDim.x) {
    const int i = (int)(idx / a.n_rec), j = (int)(idx % a.n_rec);
    const float w0 = a.W0[(size_t)j * a.n_pre + i];
    float wn = w0;
    if (!(a.recurrent && i == a.n_inl + j)) {
      double g = 0.0;
      for (int sp = 0; sp < a.n_split; ++sp) g += a.acc[sp * a.acc_stride + (size_t)i * a.ldj + j];
      wn = on_grid((double)w0 - a.lr * g);
    }
    a.Wt[(size_t)i * a.ldw + j] = wn;
    const float k = wn * 16384.0f;
    const bool exact = k == rintf(k) && fabsf(k) <= 32767.0f;
    if (!exact) a.ok[0] = 0;   // every thread that finds one writes the same value
    else kmax = max(kmax, (int)fabsf(k));
    a.W16[(size_t)i * (a.qn * kFwdThreads) + fwd_position(j, a.qn)] =
        exact ? (int16_t)k : (int16_t)0;
  }
  max_k(a.ok, kmax);
}

// One thread per (j, k): WoutT[j][k].
__global__ __launch_bounds__(256) void online_wout_kernel(OnlineArgs a) {
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)a.n_rec * a.K) return;
  const int j = (int)(idx / a.K), k = (int)(idx % a.K);
  const double g = a.accout[(size_t)k * a.ld_acc + j];
  a.WoutT[(size_t)j * a.ldk + k] = on_grid((double)a.Wout0[(size_t)k * a.n_rec + j] - a.lr * g);
}

__global__ __launch_bounds__(256) void unpack_kernel(const float* Wt, int ldw, const float* WoutT,
                                                     int ldk, int n_rec, int n_pre, int K, float* W,
                                                     float* Wout) {
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long nw = (long long)n_rec * n_pre;
  if (idx < nw) {
    const int j = (int)(idx / n_pre), i = (int)(idx % n_pre);
    W[idx] = Wt[(size_t)i * ldw + j];
  } else if (idx < nw + (long long)K * n_rec) {
    const long long r = idx - nw;
    const int k = (int)(r / n_rec), j = (int)(r % n_rec);
    Wout[r] = WoutT[(size_t)j * ldk + k];
  }
}

__global__ void set_flag_kernel(int* flag, int value) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    flag[0] = value;
    flag[1] = 0;
  }
}

// 16-byte stores over the aligned body, byte stores over the ragged ends;
// grid-stride, so any grid size covers the range.
__global__ __launch_bounds__(256) void zero_kernel(unsigned char* p, size_t bytes) {
  const size_t head = min(bytes, (size_t)((16 - ((uintptr_t)p & 15)) & 15));
  const size_t nvec = (bytes - head) / 16;
  const size_t tail0 = head + nvec * 16;
  const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t nth = (size_t)gridDim.x * blockDim.x;
  u32x4* body = (u32x4*)(p + head);
  for (size_t k = tid; k < nvec; k += nth) body[k] = u32x4{0u, 0u, 0u, 0u};
  if (tid < head) p[tid] = 0;
  if (tid < bytes - tail0) p[tail0 + tid] = 0;
}

// Several ranges in one launch: blockIdx.y picks the range, the x blocks
// stride over it as zero_kernel's do.
__global__ __launch_bounds__(256) void zero_many_kernel(ZeroRanges r) {
  const int k = blockIdx.y;
  unsigned char* p = (unsigned char*)r.p[k];
  const size_t bytes = r.bytes[k];
  const size_t head = min(bytes, (size_t)((16 - ((uintptr_t)p & 15)) & 15));
  const size_t nvec = (bytes - head) / 16;
  const size_t tail0 = head + nvec * 16;
  const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t nth = (size_t)gridDim.x * blockDim.x;
  u32x4* body = (u32x4*)(p + head);
  for (size_t q = tid; q < nvec; q += nth) body[q] = u32x4{0u, 0u, 0u, 0u};
  if (tid < head) p[tid] = 0;
  if (tid < bytes - tail0) p[tail0 + tid] = 0;
}

__global__ __launch_bounds__(256) void pack_kernel(const float* src, int rows, int cols, float* dst,
                                                   int ldd, int dst_rows, int transpose) {
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)dst_rows * ldd) return;
  const int r = (int)(idx / ldd), c = (int)(idx % ldd);
  float v = 0.0f;
  if (!transpose) {
    if (r < rows && c < cols) v = src[(size_t)r * cols + c];
  } else {
    if (r < cols && c < rows) v = src[(size_t)c * cols + r];
  }
  dst[idx] = v;
}

}  // namespace

// ---------------------------------------------------------------- launchers
// gfx950 gives a workgroup up to the whole 160 KiB of shared memory, but
// more than 64 KiB must be requested per kernel.  Each kernel is granted its
// largest size once per process (std::call_once: contexts may launch from
// several host threads), and every launch checks the outcome.
constexpr int kMaxSmem = 160 * 1024;
template <auto Kernel>   // one instance (and one flag) per kernel
hipError_t grant_smem(int bytes) {
  static std::once_flag once;
  static hipError_t result = hipSuccess;
  std::call_once(once, [bytes] {
    result = hipFuncSetAttribute(reinterpret_cast<const void*>(Kernel),
                                 hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  });
  return result;
}

template <int QN, int NL, bool SVC>
hipError_t launch_forward_qn(const FwdArgs& a, hipStream_t s) {
  if (a.smem > (size_t)kMaxSmem) return hipErrorInvalidValue;
  hipError_t e = grant_smem<&forward_kernel<QN, NL, SVC>>(kMaxSmem);
  if (e != hipSuccess) return e;
  forward_kernel<QN, NL, SVC><<<a.B, SVC ? kFwdThreads + 64 : kFwdThreads, a.smem, s>>>(a);
  return hipGetLastError();
}

template <int QN, int NL>
hipError_t launch_forward_svc(const FwdArgs& a, hipStream_t s) {
  // up to two neurons per thread: always with the service wave; more:
  // without (a ninth wave puts three waves on one SIMD, and with more than
  // about 112 registers per wave an eligibility workgroup no longer fits
  // beside the forward on its compute unit)
  if constexpr (QN <= 2)
    return a.svc ? launch_forward_qn<QN, NL, true>(a, s) : hipErrorInvalidValue;
  else
    return a.svc ? hipErrorInvalidValue : launch_forward_qn<QN, NL, false>(a, s);
}

hipError_t launch_forward(const FwdArgs& a, hipStream_t s) {
  const int qn = forward_qn(a.n_rec);
  if (a.svc && qn > 2) return hipErrorInvalidValue;
  const bool two = a.n_layers > 1;
  switch (qn) {
    case 1: return two ? launch_forward_svc<1, 2>(a, s) : launch_forward_svc<1, 1>(a, s);
    case 2: return two ? launch_forward_svc<2, 2>(a, s) : launch_forward_svc<2, 1>(a, s);
    case 4: return two ? launch_forward_svc<4, 2>(a, s) : launch_forward_svc<4, 1>(a, s);
    case 8: return two ? launch_forward_svc<8, 2>(a, s) : launch_forward_svc<8, 1>(a, s);
    case 16: return two ? launch_forward_svc<16, 2>(a, s) : launch_forward_svc<16, 1>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_input_drive(const InputArgs& a, hipStream_t s) {
  if (a.steps <= 0 || a.n_in <= 0) return hipSuccess;
  // one wave per (step, batch element) and slice of 64 kInPW positions
  static_assert(kFwdThreads / (64 * kInPW) == 1, "a slice per neuron per thread");
  const long long waves = (long long)a.steps * a.B * a.qn;
  if (waves >= (1ll << 31) || (a.qn & (a.qn - 1)) != 0) return hipErrorInvalidValue;
  input_drive_kernel<<<cdiv(waves, 4), 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_input_filter(const InputArgs& a, hipStream_t s) {
  if (a.steps <= 0 || a.n_in <= 0) return hipSuccess;
  dim3 grid(cdiv(cdiv(a.n_in, 4), 256), a.B);
  input_filter_kernel<<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_gemm_nt(const GemmArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.N, 128), cdiv(a.M, 32), a.splits);
  gemm_nt_kernel<<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_gemm_tn(const GemmArgs& a, hipStream_t s) {
  // A provides round_up(M, 16) columns; larger M in groups of 64 rows
  if (a.M > 64) {
    for (int m0 = 0; m0 < a.M; m0 += 64) {
      GemmArgs b = a;
      b.A = a.A + m0;
      b.C = a.C + (size_t)m0 * a.ldc;
      b.M = std::min(64, a.M - m0);
      hipError_t e = launch_gemm_tn(b, s);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  dim3 grid(cdiv(a.N, 128), 1, a.splits);
  const int mb = (a.M + 15) / 16;
  if (mb <= 1) gemm_tn_kernel<1><<<grid, 256, 0, s>>>(a);
  else if (mb == 2) gemm_tn_kernel<2><<<grid, 256, 0, s>>>(a);
  else if (mb == 3) gemm_tn_kernel<3><<<grid, 256, 0, s>>>(a);
  else gemm_tn_kernel<4><<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_accumulate(const float* part, int splits, size_t split_stride, int M, int N,
                             double* acc, int ld_acc, int first, hipStream_t s) {
  accumulate_kernel<<<cdiv((long long)M * N, 256), 256, 0, s>>>(part, splits, split_stride, M, N,
                                                               acc, ld_acc, first);
  return hipGetLastError();
}

hipError_t launch_coef(const CoefArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.n_post, 256), a.B);
  if (a.model == 1)
    coef_rt_kernel<GenAdjoint><<<grid, 256, 0, s>>>(a);
  else if (a.reset_through)
    coef_rt_kernel<Adjoint><<<grid, 256, 0, s>>>(a);
  else
    coef_kernel<<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

template <bool RT, int NCH>
hipError_t launch_trace_variant(const TraceArgs& a, hipStream_t s) {
  // more than 64 KiB of shared memory must be requested per kernel
  constexpr size_t smem = kTraceSmemOf(RT);
  hipError_t e = grant_smem<&trace_kernel<RT, NCH>>((int)smem);
  if (e != hipSuccess) return e;
  // eight XCDs times the groups per XCD times the row tiles of a group
  const long long wgs = 8ll * cdiv(a.n_jt * a.n_split, 8) * (a.n_pre_pad / kTileI);
  if (wgs > 0x7fffffffll) return hipErrorInvalidValue;
  // the scalar planes are addressed by 32-bit offsets within one buffer
  if ((unsigned long long)(RT ? kScalarPlanesRT : kScalarPlanes) * a.B * a.ldc * 4ull > 0xffffffffull)
    return hipErrorInvalidValue;
  trace_kernel<RT, NCH><<<dim3((unsigned)wgs), 256, smem, s>>>(a);
  return hipGetLastError();
}

template <bool RT, int... I>
hipError_t launch_trace_nch(const TraceArgs& a, hipStream_t s, std::integer_sequence<int, I...>) {
  using Fn = hipError_t (*)(const TraceArgs&, hipStream_t);
  static constexpr Fn table[] = {&launch_trace_variant<RT, I + 1>...};
  return table[(a.kpad >> 4) - 1](a, s);
}

hipError_t launch_trace(const TraceArgs& a, hipStream_t s) {
  // one kernel per chunk count of a block (kKC of them)
  if (a.kpad < kChunk || a.kpad > kBlockSteps || a.kpad % kChunk != 0) return hipErrorInvalidValue;
  const auto nch = std::make_integer_sequence<int, kKC>{};
  return a.reset_through ? launch_trace_nch<true>(a, s, nch) : launch_trace_nch<false>(a, s, nch);
}

hipError_t launch_readout(const ReadoutArgs& r, hipStream_t s) {
  if (r.n_layers < 1 || r.n_layers > 2) return hipErrorInvalidValue;
  long long gx = 1, gy = 1;
  for (int l = 0; l < r.n_layers; ++l) {
    const GradsArgs& a = r.g[l];
    gx = std::max<long long>(gx, std::max<long long>(cdiv(a.n_pre, 32), cdiv((long long)a.K * a.n_post, 256)));
    gy = std::max<long long>(gy, cdiv(a.n_post, 32));
  }
  const unsigned gz = 2 * r.n_layers + (r.loss ? 1 : 0);
  readout_kernel<<<dim3((unsigned)gx, (unsigned)gy, gz), 256, 0, s>>>(r);
  return hipGetLastError();
}

int forward_qn(int n_rec) {
  const int qn = (n_rec + kFwdThreads - 1) / kFwdThreads;
  int p = 1;
  while (p < qn) p *= 2;
  return p;
}

hipError_t launch_pack16(const float* W, int n_rec, int n_pre, int16_t* W16, int qn, int* ok,
                         hipStream_t s) {
  const long long n = (long long)n_rec * n_pre;
  pack16_kernel<<<std::min(kPackBlocks, cdiv(n, 256)), 256, 0, s>>>(W, n_rec, n_pre, W16, qn, ok);
  return hipGetLastError();
}

hipError_t launch_online_update(const OnlineArgs& a, hipStream_t s) {
  online_w_kernel<<<std::min(kPackBlocks, cdiv((long long)a.n_rec * a.n_pre, 256)), 256, 0, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  online_wout_kernel<<<cdiv((long long)a.n_rec * a.K, 256), 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_unpack_weights(const float* Wt, int ldw, const float* WoutT, int ldk, int n_rec,
                                 int n_pre, int K, float* W, float* Wout, hipStream_t s) {
  const long long n = (long long)n_rec * n_pre + (long long)K * n_rec;
  unpack_kernel<<<cdiv(n, 256), 256, 0, s>>>(Wt, ldw, WoutT, ldk, n_rec, n_pre, K, W, Wout);
  return hipGetLastError();
}

hipError_t launch_set_flag(int* flag, int value, hipStream_t s) {
  set_flag_kernel<<<1, 64, 0, s>>>(flag, value);
  return hipGetLastError();
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  const long long blocks = std::min<long long>(8192, std::max<long long>(1, cdiv((long long)(bytes / 16), 256)));
  zero_kernel<<<(int)blocks, 256, 0, s>>>((unsigned char*)p, bytes);
  return hipGetLastError();
}

hipError_t launch_zero_many(const ZeroRanges& r, hipStream_t s) {
  if (r.n < 1 || r.n > ZeroRanges::kMax) return hipErrorInvalidValue;
  long long blocks = 1;
  for (int k = 0; k < r.n; ++k)
    blocks = std::max<long long>(blocks, std::min<long long>(8192, cdiv((long long)(r.bytes[k] / 16), 256)));
  zero_many_kernel<<<dim3((unsigned)blocks, (unsigned)r.n), 256, 0, s>>>(r);
  return hipGetLastError();
}

hipError_t launch_pack(const float* src, int rows, int cols, float* dst, int ldd, int dst_rows,
                       int transpose, hipStream_t s) {
  const long long n = (long long)dst_rows * ldd;
  pack_kernel<<<cdiv(n, 256), 256, 0, s>>>(src, rows, cols, dst, ldd, dst_rows, transpose);
  return hipGetLastError();
}

}  // namespace eprop
