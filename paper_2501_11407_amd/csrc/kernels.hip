// gfx950 kernels of the online e-prop step.
//
// Built with -ffp-contract=off: every a*b+c written below is a rounded
// multiply followed by a rounded add unless fmaf/fma is spelled out.  The
// forward kernel relies on this to reproduce fp32 spike decisions operation
// by operation; the eligibility kernel uses explicit fused multiply-adds where
// precision only gains from them.
#include "kernels.h"

#include <math.h>

namespace eprop {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ inline int lanes_below(unsigned long long m, int lane) {
  return __popcll(m & ((1ull << lane) - 1ull));
}

__device__ inline f32x4 load_nt(const float* p) {
  return __builtin_nontemporal_load((const f32x4*)p);
}
__device__ inline void store_nt(float* p, f32x4 v) { __builtin_nontemporal_store(v, (f32x4*)p); }

inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

// ---------------------------------------------------------------- forward
// One workgroup per batch element runs `steps` timesteps of every layer; the
// neuron state of the threads' neurons stays in registers, the filtered
// presynaptic vector and the readout in shared memory.  Per step and layer:
//   1. p = [in ; z_prev]; zbar = alpha*zbar + p; each wave lists the indices
//      of its contiguous slice of p that are 1, in ascending order.
//   2. drive I_j = sum of W_ji over the listed i, visited in ascending i (the
//      order of a plain sequential sum), then the neuron step with one
//      rounding per operation:
//        v = alpha*v; v = v + I; v = v - thr*z_prev
//        a = rho*a;   a = a + z_prev
//        A = beta_j*a; A = thr + A;  x = v - A;  z = x > 0
//        psi = (gamma/thr) * max(0, 1 - |x|/thr)
//   3. readout y = kappa*y + W_out z (over the spiking neurons), softmax,
//      delta = softmax - onehot(label), cross-entropy into the loss;
//   4. ztilde = kappa*ztilde + z.
// The learning signal L = W_out^T delta is one GEMM over the whole block.
struct FwdLds {
  int* act; int* spk; int* cnt; float* red; float* sy; float* szb; uint8_t* zc; uint8_t* xs;
  int rwmax, npad;
};

template <int QN, int LI>
__device__ __forceinline__ void forward_layer_step(const FwdArgs& A, const FwdLds& S, int t, int b,
                                                   int cur, float (&v)[QN], float (&ad)[QN],
                                                   float (&zt)[QN], double& loss) {
  const FwdLayer& Ly = A.L[LI];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const uint8_t* zprev = S.zc + (LI * 2 + cur) * S.npad;
  uint8_t* znow = S.zc + (LI * 2 + (cur ^ 1)) * S.npad;
  const uint8_t* inp;
  if constexpr (LI == 0)
    inp = S.xs + (t % kFwdXSteps) * A.n_in;      // staged input spikes of this step
  else
    inp = S.zc + ((LI - 1) * 2 + (cur ^ 1)) * S.npad;
  float* szb = S.szb + (LI == 0 ? 0 : A.L[0].n_pre);
  float* sy = S.sy + LI * A.K_out;
  const size_t row = (size_t)t * A.Bp + b;

  // 1. presynaptic vector, its filter, ordered active lists
  const int rw = Ly.rows_per_wave;
  const int i_beg = w * rw, i_end = min(Ly.n_pre, i_beg + rw);
  float* zbk = Ly.zbarK + ((size_t)b * A.Kmax + t) * Ly.ldi;
  int n_act = 0;
  for (int base = i_beg; base < i_end; base += kWave) {
    const int i = base + lane;
    bool on = false;
    if (i < i_end) {
      const uint8_t sv = (i < Ly.n_inl) ? inp[i] : zprev[i - Ly.n_inl];
      on = sv != 0;
      const float zv = A.alpha * szb[i] + (on ? 1.0f : 0.0f);
      szb[i] = zv;
      zbk[i] = zv;
    }
    const unsigned long long m = __ballot(on);
    if (on) S.act[w * S.rwmax + n_act + lanes_below(m, lane)] = i;
    n_act += __popcll(m);
  }
  if (lane == 0) S.cnt[w] = n_act;
  __syncthreads();

  // 2. drive and neuron step.  Rows of Wt are padded to a multiple of the
  // workgroup size; chunks q with q*kFwdThreads >= n_rec are skipped (QN is
  // rounded up to a power of two).
  float I[QN];
#pragma unroll
  for (int q = 0; q < QN; ++q) I[q] = 0.0f;
  for (int ww = 0; ww < kFwdWaves; ++ww) {
    const int c = S.cnt[ww];
    const int* lst = S.act + ww * S.rwmax;
#pragma unroll 4
    for (int k = 0; k < c; ++k) {
      const float* wrow = Ly.Wt + (size_t)lst[k] * Ly.ldw + tid;
#pragma unroll
      for (int q = 0; q < QN; ++q)
        if (q * kFwdThreads < A.n_rec) I[q] += wrow[q * kFwdThreads];
    }
  }
  int n_spk = 0;
#pragma unroll
  for (int q = 0; q < QN; ++q) {
    const int j = q * kFwdThreads + tid;
    bool z = false;
    if (j < A.n_rec) {
      const float zp = zprev[j] ? 1.0f : 0.0f;
      float vv = A.alpha * v[q];
      vv = vv + I[q];
      vv = vv - A.thr * zp;
      float aa = A.rho * ad[q];
      aa = aa + zp;
      const float bj = (j < A.n_adaptive) ? A.beta : 0.0f;
      float th = bj * aa;
      th = A.thr + th;
      const float x = vv - th;
      v[q] = vv;
      ad[q] = aa;
      z = x > 0.0f;
      znow[j] = z ? 1 : 0;
      const float u = 1.0f - fabsf(x) / A.thr;
      Ly.psiK[row * A.ldj + j] = A.gamma_over_thr * fmaxf(u, 0.0f);
    }
    const unsigned long long m = __ballot(z);
    if (z) S.spk[w * A.jlist + n_spk + lanes_below(m, lane)] = j;
    n_spk += __popcll(m);
    if (A.spikes) {
      const int w0 = (q * kFwdThreads + w * kWave) >> 5;
      uint32_t* srow = A.spikes + (((size_t)t * A.n_layers + LI) * A.B + b) * A.W32;
      if (lane == 0 && w0 < A.W32) srow[w0] = (uint32_t)m;
      if (lane == 1 && w0 + 1 < A.W32) srow[w0 + 1] = (uint32_t)(m >> 32);
    }
  }
  if (lane == 0) S.cnt[kFwdWaves + w] = n_spk;
  __syncthreads();

  // 3. readout (rows of the transposed readout weights of the spiking
  // neurons, read coalesced over k), softmax cross-entropy
  for (int k = tid; k < A.K_out; k += kFwdThreads) {
    float Y = 0.0f;
    for (int ww = 0; ww < kFwdWaves; ++ww) {
      const int c = S.cnt[kFwdWaves + ww];
      const int* lst = S.spk + ww * A.jlist;
#pragma unroll 8
      for (int s = 0; s < c; ++s) Y += Ly.WoutT[(size_t)lst[s] * A.ldk + k];
    }
    float yy = A.kappa * sy[k];
    yy = yy + Y;
    sy[k] = yy;
  }
  __syncthreads();
  const int label = A.labels[b];
  const bool label_ok = label >= 0 && label < A.K_out;
  if (w == 0) {
    float m = -INFINITY;
    for (int k = lane; k < A.K_out; k += kWave) m = fmaxf(m, sy[k]);
    m = wave_max(m);
    float se = 0.0f;
    for (int k = lane; k < A.K_out; k += kWave) se += expf(sy[k] - m);
    se = wave_sum(se);
    if (lane == 0) {
      S.red[0] = m;
      S.red[1] = se;
      if (label_ok)
        loss += log((double)se) - ((double)sy[label] - (double)m);
      else
        *A.err_flag = 1;
    }
  }
  __syncthreads();
  {
    const float m = S.red[0], se = S.red[1];
    for (int k = tid; k < A.K_out; k += kFwdThreads) {
      const float d = expf(sy[k] - m) / se - ((k == label) ? 1.0f : 0.0f);
      Ly.deltaK[row * A.ldk + k] = d;
    }
  }

  // 4. filtered spikes
#pragma unroll
  for (int q = 0; q < QN; ++q) {
    const int j = q * kFwdThreads + tid;
    if (j < A.n_rec) {
      float zz = A.kappa * zt[q];
      zz = zz + (znow[j] ? 1.0f : 0.0f);
      zt[q] = zz;
      Ly.ztK[row * A.ldn + j] = zz;
    }
  }
  __syncthreads();
}

template <int QN, int LI>
__device__ __forceinline__ void forward_state(const FwdArgs& A, const FwdLds& S, int b, bool load,
                                              float (&v)[QN], float (&ad)[QN], float (&zt)[QN],
                                              int cur) {
  const FwdLayer& Ly = A.L[LI];
  const int tid = threadIdx.x;
  float* szb = S.szb + (LI == 0 ? 0 : A.L[0].n_pre);
  float* sy = S.sy + LI * A.K_out;
  uint8_t* zc = S.zc + (LI * 2 + cur) * S.npad;
#pragma unroll
  for (int q = 0; q < QN; ++q) {
    const int j = q * kFwdThreads + tid;
    if (j < A.n_rec) {
      const size_t o = (size_t)b * A.n_rec + j;
      if (load) {
        v[q] = Ly.v[o]; ad[q] = Ly.a[o]; zt[q] = Ly.ztil[o]; zc[j] = Ly.z[o];
      } else {
        Ly.v[o] = v[q]; Ly.a[o] = ad[q]; Ly.ztil[o] = zt[q]; Ly.z[o] = zc[j];
      }
    }
  }
  for (int i = tid; i < Ly.n_pre; i += kFwdThreads) {
    if (load) szb[i] = Ly.zbar[(size_t)b * Ly.n_pre + i];
    else Ly.zbar[(size_t)b * Ly.n_pre + i] = szb[i];
  }
  for (int k = tid; k < A.K_out; k += kFwdThreads) {
    if (load) sy[k] = Ly.y[(size_t)b * A.K_out + k];
    else Ly.y[(size_t)b * A.K_out + k] = sy[k];
  }
}

template <int QN>
__global__ __launch_bounds__(kFwdThreads) void forward_kernel(FwdArgs A) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int b = blockIdx.x;
  FwdLds S;
  S.rwmax = A.L[0].rows_per_wave;
  if (A.n_layers > 1) S.rwmax = max(S.rwmax, A.L[1].rows_per_wave);
  S.npad = (A.n_rec + 3) & ~3;
  S.act = (int*)smem;                          // [waves][rwmax]
  S.spk = S.act + kFwdWaves * S.rwmax;         // [waves][jlist]
  S.cnt = S.spk + kFwdWaves * A.jlist;         // [2 * waves]
  S.red = (float*)(S.cnt + 2 * kFwdWaves);     // [2]
  S.sy = S.red + 2;                            // [n_layers][K_out]
  S.szb = S.sy + A.n_layers * A.K_out;         // [n_pre_0 + n_pre_1]
  const int npre_total = A.L[0].n_pre + (A.n_layers > 1 ? A.L[1].n_pre : 0);
  S.zc = (uint8_t*)(S.szb + npre_total);       // [n_layers][2][npad]
  S.xs = S.zc + A.n_layers * 2 * S.npad;       // [kFwdXSteps][n_in]

  float v0[QN], a0[QN], zt0[QN], v1[QN], a1[QN], zt1[QN];
  forward_state<QN, 0>(A, S, b, true, v0, a0, zt0, 0);
  if (A.n_layers > 1) forward_state<QN, 1>(A, S, b, true, v1, a1, zt1, 0);
  double loss0 = 0.0, loss1 = 0.0;
  int cur = 0;
  __syncthreads();
  for (int t = 0; t < A.steps; ++t) {
    if (t % kFwdXSteps == 0) {
      // stage the input spikes of the next kFwdXSteps steps (one round trip)
      const int ns = min(kFwdXSteps, A.steps - t);
#pragma unroll
      for (int tt = 0; tt < kFwdXSteps; ++tt) {
        if (tt < ns) {
          const uint8_t* xrow = A.x + ((size_t)(t + tt) * A.B + b) * A.n_in;
          for (int i = threadIdx.x; i < A.n_in; i += kFwdThreads) S.xs[tt * A.n_in + i] = xrow[i];
        }
      }
      __syncthreads();
    }
    forward_layer_step<QN, 0>(A, S, t, b, cur, v0, a0, zt0, loss0);
    if (A.n_layers > 1) forward_layer_step<QN, 1>(A, S, t, b, cur, v1, a1, zt1, loss1);
    cur ^= 1;
  }
  forward_state<QN, 0>(A, S, b, false, v0, a0, zt0, cur);
  if (A.n_layers > 1) forward_state<QN, 1>(A, S, b, false, v1, a1, zt1, cur);
  if (threadIdx.x == 0) {
    A.L[0].lossacc[b] += loss0;
    if (A.n_layers > 1) A.L[1].lossacc[b] += loss1;
  }
}

// ---------------------------------------------------------------- MFMA GEMM
// v_mfma_f32_16x16x4f32 operand layout (64 lanes, lane = r + 16*g):
//   A[16 x 4]:  lane holds A[r][g];  B[4 x 16]: lane holds B[g][r];
//   D[16 x 16]: lane holds D[4*g + q][r] in accumulator register q.
// Each lane loads 4 consecutive k (float4) of its row of A and of Bm and feeds
// them to 4 MFMAs; both operands use the same k permutation, so the 4 MFMAs
// together contract 16 consecutive k.  One wave computes a 32x32 tile
// (2x2 blocks of 16x16); a block of 4 waves covers 32 (m) x 128 (n).
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

// Same tiling with both operands stored k-major: lane (r, g) takes
// A[k][m0 + r] and Bm[k][n0 + r] for its four k of every 16-k chunk.
__global__ __launch_bounds__(256) void gemm_tn_kernel(GemmArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int m0 = blockIdx.y * 32;
  const int n0 = (blockIdx.x * 4 + wave) * 32;
  if (n0 >= a.N) return;
  const int split = blockIdx.z;
  const int kb = split * a.k_chunk;
  const int ke = min(a.K, kb + a.k_chunk);
  const int r = lane & 15, g = lane >> 4;
  f32x4 c00 = {0.f, 0.f, 0.f, 0.f}, c01 = c00, c10 = c00, c11 = c00;
  for (int k = kb; k < ke; k += 16) {
    f32x4 va0, va1, vb0, vb1;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const size_t kk = (size_t)(k + 4 * g + q);
      va0[q] = a.A[kk * a.lda + m0 + r];
      va1[q] = a.A[kk * a.lda + m0 + 16 + r];
      vb0[q] = a.Bm[kk * a.ldb + n0 + r];
      vb1[q] = a.Bm[kk * a.ldb + n0 + 16 + r];
    }
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

// Split-K partials added into an fp64 accumulator in split order.
__global__ __launch_bounds__(256) void accumulate_kernel(const float* part, int splits, size_t ss,
                                                        int M, int N, double* acc, int ld, int first) {
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)M * N) return;
  const int m = (int)(idx / N), n = (int)(idx % N);
  double s = first ? 0.0 : acc[(size_t)m * ld + n];
  for (int sp = 0; sp < splits; ++sp) s += (double)part[sp * ss + (size_t)m * N + n];
  acc[(size_t)m * ld + n] = s;
}

// ---------------------------------------------------------------- eligibility
// A workgroup owns one 256-wide segment of postsynaptic neurons and a group
// of presynaptic rows; lane l of every wave owns the four neurons
// j0 = seg*256 + 4l..4l+3 and wave w rows ib + w*R .. ib + w*R + R-1.
// Segments holding adaptive neurons move two trace arrays per synapse and use
// R = 2 rows per thread, LIF segments one array and R = 4, so every wave does
// about the same arithmetic; groups of 16 rows list their adaptive and LIF
// workgroups next to each other in dispatch order.
// The workgroup walks the batch; for each batch element the traces are read
// once, advanced through the block's steps and written once.  psi and L of
// the segment and zbar of the rows are shared through shared memory,
// kTraceChunk steps at a time, in a pipeline over chunks (batch element,
// step range): the next chunk's vectors are loaded into registers and the
// next batch element's traces prefetched while the current chunk computes.
// Per step, for each (i, j):
//   e    = psi_j zbar_i - psi_j beta_j epsa      (dz_j/dW_ji)
//   ebar = kappa ebar + e                        (readout filter on the trace)
//   acc += L_j ebar                              (fp32 within a chunk, fp64 across)
//   epsa = (rho - beta_j psi_j) epsa + psi_j zbar_i   (adaptive j)
// On LIF lanes of an adaptive segment beta_j = 0, so e = psi_j zbar_i exactly.
constexpr int kStage = kTraceChunk * 64 / (kTraceWaves * 64);   // float4 per thread per vector
static_assert(kStage * kTraceWaves * 64 == kTraceChunk * 64, "chunk must split evenly");
static_assert(kTraceChunk * kRowPad <= kTraceWaves * 64, "zbar chunk must fit one load per thread");

struct TraceShared {
  f32x4 ps[kTraceChunk][64];
  f32x4 lv[kTraceChunk][64];
  float zb[kTraceChunk][kRowPad];
};

struct TraceStage {
  f32x4 ps[kStage], lv[kStage];
  float zb;
};

// Every lane issues the same loads whatever the chunk (indices are clamped
// to valid rows), so the number of loads in flight is the same on every path
// and waits on them never have to drain the whole queue.
template <int ROWS>
__device__ __forceinline__ void trace_stage_load(const TraceArgs& a, TraceStage& g, int b, int c0,
                                                 int nt, int seg, int ib) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int u = 0; u < kStage; ++u) {
    const int k = tid + u * kTraceWaves * 64;
    const int tt = min(k >> 6, nt - 1), l = k & 63;
    const size_t row = (size_t)(c0 + tt) * a.Bp + b;
    g.ps[u] = *(const f32x4*)(a.psiK + row * a.ldv + seg * 256 + 4 * l);
    g.lv[u] = *(const f32x4*)(a.LK + row * a.ldv + seg * 256 + 4 * l);
  }
  const int kz = tid % (kTraceChunk * ROWS);
  const int tt = min(kz / ROWS, nt - 1), r = kz % ROWS;
  g.zb = a.zbarK[((size_t)b * a.Kmax + c0 + tt) * a.ldi + ib + r];
}

template <int ROWS>
__device__ __forceinline__ void trace_stage_store(const TraceStage& g, int nt, TraceShared& S) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int u = 0; u < kStage; ++u) {
    const int k = tid + u * kTraceWaves * 64;
    const int tt = k >> 6, l = k & 63;
    if (tt < nt) {
      S.ps[tt][l] = g.ps[u];
      S.lv[tt][l] = g.lv[u];
    }
  }
  if (tid < kTraceChunk * ROWS) {
    const int tt = tid / ROWS, r = tid % ROWS;
    if (tt < nt) S.zb[tt][r] = g.zb;
  }
}

template <int R, bool ALIF, bool FIRST>
__device__ __forceinline__ void trace_body(const TraceArgs& a, TraceShared& S, int seg, int ib) {
  constexpr int ROWS = R * kTraceWaves;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int j0 = seg * 256 + lane * 4;
  const bool active = j0 < a.n_post;
  const bool has_a = ALIF && j0 < a.n_adaptive;   // lane holds eps^a
  const int i0 = ib + w * R;
  float bj[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) bj[r] = (ALIF && j0 + r < a.n_adaptive) ? a.beta : 0.0f;

  double acc[R][4];
#pragma unroll
  for (int ii = 0; ii < R; ++ii)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      acc[ii][r] = (FIRST || !active) ? 0.0 : a.acc[(size_t)(i0 + ii) * a.ldj + j0 + r];

  const size_t bs_e = (size_t)a.n_pre_pad * a.ldj;
  const size_t bs_a = (size_t)a.n_pre_pad * a.lda;
  float* pe0 = a.ebar + (size_t)i0 * a.ldj + j0;
  float* pa0 = a.epsa + (size_t)i0 * a.lda + j0;
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  const int nch = (a.steps + kTraceChunk - 1) / kTraceChunk;
  const int total = a.B * nch;

  f32x4 E[R], Aa[ALIF ? R : 1], En[R], An[ALIF ? R : 1];
#pragma unroll
  for (int ii = 0; ii < R; ++ii) {
    E[ii] = zero;
    En[ii] = zero;
    if (!FIRST && active) E[ii] = load_nt(pe0 + (size_t)ii * a.ldj);
  }
  if constexpr (ALIF) {
#pragma unroll
    for (int ii = 0; ii < R; ++ii) {
      Aa[ii] = zero;
      An[ii] = zero;
      if (!FIRST && has_a) Aa[ii] = load_nt(pa0 + (size_t)ii * a.lda);
    }
  }
  TraceStage g;
  trace_stage_load<ROWS>(a, g, 0, 0, min(kTraceChunk, a.steps), seg, ib);
  trace_stage_store<ROWS>(g, min(kTraceChunk, a.steps), S);
  __syncthreads();

  for (int q = 0; q < total; ++q) {
    const int b = q / nch, c = q - b * nch;
    const int nt = min(kTraceChunk, a.steps - c * kTraceChunk);
    // Order of issue: next batch element's traces (during its last chunk),
    // then the next chunk's shared vectors.
    if (!FIRST && c == nch - 1 && b + 1 < a.B) {
#pragma unroll
      for (int ii = 0; ii < R; ++ii)
        if (active) En[ii] = load_nt(pe0 + (size_t)(b + 1) * bs_e + (size_t)ii * a.ldj);
      if constexpr (ALIF) {
#pragma unroll
        for (int ii = 0; ii < R; ++ii)
          if (has_a) An[ii] = load_nt(pa0 + (size_t)(b + 1) * bs_a + (size_t)ii * a.lda);
      }
    }
    const int qn = min(q + 1, total - 1);
    const int nb = qn / nch, nc = qn - nb * nch;
    const int nnt = min(kTraceChunk, a.steps - nc * kTraceChunk);
    trace_stage_load<ROWS>(a, g, nb, nc * kTraceChunk, nnt, seg, ib);

    // L * ebar summed over the chunk in fp32, then added to the fp64 accumulator
    float part[R][4];
#pragma unroll
    for (int ii = 0; ii < R; ++ii)
#pragma unroll
      for (int r = 0; r < 4; ++r) part[ii][r] = 0.0f;
    for (int tt = 0; tt < nt; ++tt) {
      const f32x4 ps = S.ps[tt][lane];
      const f32x4 lv = S.lv[tt][lane];
      float zb[R];
#pragma unroll
      for (int ii = 0; ii < R; ++ii) zb[ii] = S.zb[tt][w * R + ii];
      if constexpr (ALIF) {
        float pb[4], rb[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          pb[r] = ps[r] * bj[r];
          rb[r] = a.rho - pb[r];
        }
#pragma unroll
        for (int ii = 0; ii < R; ++ii)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float pz = ps[r] * zb[ii];
            const float e = fmaf(-pb[r], Aa[ii][r], pz);
            E[ii][r] = fmaf(a.kappa, E[ii][r], e);
            Aa[ii][r] = fmaf(rb[r], Aa[ii][r], pz);
            part[ii][r] = fmaf(lv[r], E[ii][r], part[ii][r]);
          }
      } else {
#pragma unroll
        for (int ii = 0; ii < R; ++ii)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            E[ii][r] = fmaf(a.kappa, E[ii][r], ps[r] * zb[ii]);
            part[ii][r] = fmaf(lv[r], E[ii][r], part[ii][r]);
          }
      }
    }
#pragma unroll
    for (int ii = 0; ii < R; ++ii)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[ii][r] += (double)part[ii][r];

    if (c == nch - 1) {
#pragma unroll
      for (int ii = 0; ii < R; ++ii) {
        if (active) store_nt(pe0 + (size_t)b * bs_e + (size_t)ii * a.ldj, E[ii]);
        E[ii] = En[ii];
      }
      if constexpr (ALIF) {
#pragma unroll
        for (int ii = 0; ii < R; ++ii) {
          if (has_a) store_nt(pa0 + (size_t)b * bs_a + (size_t)ii * a.lda, Aa[ii]);
          Aa[ii] = An[ii];
        }
      }
    }
    __syncthreads();   // every wave is done with this chunk's shared vectors
    if (q + 1 < total) trace_stage_store<ROWS>(g, nnt, S);
    __syncthreads();
  }
  if (active) {
#pragma unroll
    for (int ii = 0; ii < R; ++ii)
#pragma unroll
      for (int r = 0; r < 4; ++r) a.acc[(size_t)(i0 + ii) * a.ldj + j0 + r] = acc[ii][r];
  }
}

// Block index -> (row group of kRowPad rows, kind, segment): per group, two
// adaptive workgroups of kRowPad/2 rows per adaptive segment, then one LIF
// workgroup of kRowPad rows per LIF segment.
template <bool FIRST>
__global__ __launch_bounds__(kTraceWaves * 64) void trace_kernel(TraceArgs a) {
  __shared__ TraceShared S;
  const int per_group = 2 * a.n_seg_a + a.n_seg_l;
  const int grp = blockIdx.x / per_group, k = blockIdx.x - grp * per_group;
  if (k < 2 * a.n_seg_a)
    trace_body<kRowPad / (2 * kTraceWaves), true, FIRST>(a, S, k >> 1,
                                                         grp * kRowPad + (k & 1) * (kRowPad / 2));
  else
    trace_body<kRowPad / kTraceWaves, false, FIRST>(a, S, a.n_seg_a + (k - 2 * a.n_seg_a),
                                                    grp * kRowPad);
}

// ---------------------------------------------------------------- gradient read-out
// 32x32 tiles through shared memory: acc is [i][j], dW is [j][i].
__global__ __launch_bounds__(256) void grads_kernel(GradsArgs a) {
  __shared__ double tile[32][33];
  const int i0 = blockIdx.x * 32, j0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;   // 32 x 8
  for (int yy = ty; yy < 32; yy += 8) {
    const int i = i0 + yy, j = j0 + tx;
    tile[yy][tx] = (a.valid && i < a.n_pre && j < a.n_post) ? a.acc[(size_t)i * a.ldj + j] : 0.0;
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

__global__ __launch_bounds__(256) void grads_out_kernel(GradsArgs a) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const int k = blockIdx.y;
  if (j >= a.n_post) return;
  a.dWout[(size_t)k * a.n_post + j] = a.valid ? (float)a.accout[(size_t)k * a.ld_acc + j] : 0.0f;
}

// One thread: a fixed summation order over layers and batch elements.
__global__ void loss_kernel(const double* lossacc, int B, int n_layers, size_t layer_stride,
                            double* out) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  double s = 0.0;
  for (int l = 0; l < n_layers; ++l)
    for (int b = 0; b < B; ++b) s += lossacc[(size_t)l * layer_stride + b];
  *out = s;
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
template <int QN>
hipError_t launch_forward_qn(const FwdArgs& a, hipStream_t s) {
  // gfx950 gives a workgroup up to the whole 160 KiB of shared memory, but
  // more than 64 KiB must be requested per kernel.
  static size_t granted = 64 * 1024;
  if (a.smem > granted) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&forward_kernel<QN>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)a.smem);
    if (e != hipSuccess) return e;
    granted = a.smem;
  }
  forward_kernel<QN><<<a.B, kFwdThreads, a.smem, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_forward(const FwdArgs& a, hipStream_t s) {
  const int qn = (a.n_rec + kFwdThreads - 1) / kFwdThreads;
  if (qn <= 1) return launch_forward_qn<1>(a, s);
  if (qn <= 2) return launch_forward_qn<2>(a, s);
  if (qn <= 4) return launch_forward_qn<4>(a, s);
  if (qn <= 8) return launch_forward_qn<8>(a, s);
  if (qn <= 16) return launch_forward_qn<16>(a, s);
  return hipErrorInvalidValue;
}

hipError_t launch_gemm_nt(const GemmArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.N, 128), cdiv(a.M, 32), a.splits);
  gemm_nt_kernel<<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_gemm_tn(const GemmArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.N, 128), cdiv(a.M, 32), a.splits);
  gemm_tn_kernel<<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_accumulate(const float* part, int splits, size_t split_stride, int M, int N,
                             double* acc, int ld_acc, int first, hipStream_t s) {
  accumulate_kernel<<<cdiv((long long)M * N, 256), 256, 0, s>>>(part, splits, split_stride, M, N,
                                                               acc, ld_acc, first);
  return hipGetLastError();
}

hipError_t launch_trace(const TraceArgs& a, hipStream_t s) {
  const int groups = a.n_pre_pad / kRowPad;
  const int grid = groups * (2 * a.n_seg_a + a.n_seg_l);
  if (a.first)
    trace_kernel<true><<<grid, kTraceWaves * 64, 0, s>>>(a);
  else
    trace_kernel<false><<<grid, kTraceWaves * 64, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_grads(const GradsArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.n_pre, 32), cdiv(a.n_post, 32));
  grads_kernel<<<grid, 256, 0, s>>>(a);
  dim3 grid2(cdiv(a.n_post, 256), a.K);
  grads_out_kernel<<<grid2, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_loss(const double* lossacc, int B, int n_layers, size_t layer_stride,
                       double* out, hipStream_t s) {
  loss_kernel<<<1, 64, 0, s>>>(lossacc, B, n_layers, layer_stride, out);
  return hipGetLastError();
}

hipError_t launch_pack(const float* src, int rows, int cols, float* dst, int ldd, int dst_rows,
                       int transpose, hipStream_t s) {
  const long long n = (long long)dst_rows * ldd;
  pack_kernel<<<cdiv(n, 256), 256, 0, s>>>(src, rows, cols, dst, ldd, dst_rows, transpose);
  return hipGetLastError();
}

}  // namespace eprop
