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
// One workgroup per batch element runs `steps` timesteps of every layer.
// Per step and layer:
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
//   4. learning signal L = W_out^T delta and ztilde = kappa*ztilde + z.
__global__ __launch_bounds__(kFwdThreads) void forward_kernel(FwdArgs A) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int rwmax = A.L[0].rows_per_wave;
  if (A.n_layers > 1) rwmax = max(rwmax, A.L[1].rows_per_wave);
  int* act = (int*)smem;                 // [4][rwmax]  active presynaptic indices
  int* spk = act + 4 * rwmax;            // [4][jlist]  spiking neurons
  int* cnt = spk + 4 * A.jlist;          // [8]         list lengths
  float* sy = (float*)(cnt + 8);         // [K_out]
  float* sd = sy + A.K_out;              // [K_out]
  float* red = sd + A.K_out;             // [2]         max, sum of the softmax
  uint8_t* zc = (uint8_t*)(red + 2);     // [n_layers][2][npad] spikes at t-1 and t
  const int npad = (A.n_rec + 3) & ~3;
  const int label = A.labels[b];
  const bool label_ok = label >= 0 && label < A.K_out;
  const int QN = (A.n_rec + kFwdThreads - 1) / kFwdThreads;

  for (int l = 0; l < A.n_layers; ++l)
    for (int j = tid; j < A.n_rec; j += kFwdThreads)
      zc[(l * 2) * npad + j] = A.L[l].z[(size_t)b * A.n_rec + j];
  double loss0 = 0.0, loss1 = 0.0;
  int cur = 0;
  __syncthreads();

  for (int t = 0; t < A.steps; ++t) {
    for (int l = 0; l < A.n_layers; ++l) {
      const FwdLayer& Ly = A.L[l];
      const uint8_t* zprev = zc + (l * 2 + cur) * npad;
      uint8_t* znow = zc + (l * 2 + (cur ^ 1)) * npad;
      const uint8_t* inp = (l == 0) ? A.x + ((size_t)t * A.B + b) * A.n_in
                                    : zc + ((l - 1) * 2 + (cur ^ 1)) * npad;

      // 1. presynaptic vector, its filter, ordered active lists
      const int rw = Ly.rows_per_wave;
      const int i_beg = w * rw, i_end = min(Ly.n_pre, i_beg + rw);
      int n_act = 0;
      for (int base = i_beg; base < i_end; base += kWave) {
        const int i = base + lane;
        bool on = false;
        if (i < i_end) {
          const uint8_t sv = (i < Ly.n_inl) ? inp[i] : zprev[i - Ly.n_inl];
          on = sv != 0;
          float* zp = Ly.zbar + (size_t)b * Ly.n_pre + i;
          const float zv = A.alpha * *zp + (on ? 1.0f : 0.0f);
          *zp = zv;
          Ly.zbarK[((size_t)i * A.B + b) * A.Kmax + t] = zv;
        }
        const unsigned long long m = __ballot(on);
        if (on) act[w * rwmax + n_act + lanes_below(m, lane)] = i;
        n_act += __popcll(m);
      }
      if (lane == 0) cnt[w] = n_act;
      __syncthreads();

      // 2. drive and neuron step
      int n_spk = 0;
      for (int q = 0; q < QN; ++q) {
        const int j = q * kFwdThreads + tid;
        bool z = false;
        if (j < A.n_rec) {
          float I = 0.0f;
          for (int ww = 0; ww < 4; ++ww) {
            const int c = cnt[ww];
            const int* lst = act + ww * rwmax;
#pragma unroll 8
            for (int k = 0; k < c; ++k) I += Ly.Wt[(size_t)lst[k] * Ly.ldw + j];
          }
          const size_t o = (size_t)b * A.n_rec + j;
          const float zp = zprev[j] ? 1.0f : 0.0f;
          float v = A.alpha * Ly.v[o];
          v = v + I;
          v = v - A.thr * zp;
          float ad = A.rho * Ly.a[o];
          ad = ad + zp;
          const float bj = (j < A.n_adaptive) ? A.beta : 0.0f;
          float th = bj * ad;
          th = A.thr + th;
          const float x = v - th;
          Ly.v[o] = v;
          Ly.a[o] = ad;
          z = x > 0.0f;
          znow[j] = z ? 1 : 0;
          const float u = 1.0f - fabsf(x) / A.thr;
          Ly.psiK[((size_t)b * A.Kmax + t) * A.ldj + j] = A.gamma_over_thr * fmaxf(u, 0.0f);
        }
        const unsigned long long m = __ballot(z);
        if (z) spk[w * A.jlist + n_spk + lanes_below(m, lane)] = j;
        n_spk += __popcll(m);
        if (A.spikes) {
          const int w0 = (q * kFwdThreads + w * kWave) >> 5;
          uint32_t* row = A.spikes + (((size_t)t * A.n_layers + l) * A.B + b) * A.W32;
          if (lane == 0 && w0 < A.W32) row[w0] = (uint32_t)m;
          if (lane == 1 && w0 + 1 < A.W32) row[w0 + 1] = (uint32_t)(m >> 32);
        }
      }
      if (lane == 0) cnt[4 + w] = n_spk;
      __syncthreads();

      // 3. readout, softmax cross-entropy
      for (int k = tid; k < A.K_out; k += kFwdThreads) {
        float Y = 0.0f;
        for (int ww = 0; ww < 4; ++ww) {
          const int c = cnt[4 + ww];
          const int* lst = spk + ww * A.jlist;
          for (int s = 0; s < c; ++s) Y += Ly.Wout[(size_t)k * Ly.ldo + lst[s]];
        }
        float yy = A.kappa * Ly.y[(size_t)b * A.K_out + k];
        yy = yy + Y;
        Ly.y[(size_t)b * A.K_out + k] = yy;
        sy[k] = yy;
      }
      __syncthreads();
      if (w == 0) {
        float m = -INFINITY;
        for (int k = lane; k < A.K_out; k += kWave) m = fmaxf(m, sy[k]);
        m = wave_max(m);
        float se = 0.0f;
        for (int k = lane; k < A.K_out; k += kWave) se += expf(sy[k] - m);
        se = wave_sum(se);
        if (lane == 0) {
          red[0] = m;
          red[1] = se;
          if (label_ok) {
            const double ce = log((double)se) - ((double)sy[label] - (double)m);
            if (l == 0) loss0 += ce; else loss1 += ce;
          } else {
            *A.err_flag = 1;
          }
        }
      }
      __syncthreads();
      {
        const float m = red[0], se = red[1];
        for (int k = tid; k < A.K_out; k += kFwdThreads) {
          const float d = expf(sy[k] - m) / se - ((k == label) ? 1.0f : 0.0f);
          sd[k] = d;
          Ly.deltaK[(size_t)k * A.ldbk + (size_t)t * A.Bp + b] = d;
        }
      }
      __syncthreads();

      // 4. learning signal and filtered spikes
      for (int j = tid; j < A.n_rec; j += kFwdThreads) {
        float Lj = 0.0f;
        for (int k = 0; k < A.K_out; ++k) Lj = fmaf(Ly.Wout[(size_t)k * Ly.ldo + j], sd[k], Lj);
        Ly.LK[((size_t)b * A.Kmax + t) * A.ldj + j] = Lj;
        const size_t o = (size_t)b * A.n_rec + j;
        float zt = A.kappa * Ly.ztil[o];
        zt = zt + (znow[j] ? 1.0f : 0.0f);
        Ly.ztil[o] = zt;
        Ly.ztK[(size_t)j * A.ldbk + (size_t)t * A.Bp + b] = zt;
      }
      __syncthreads();
    }
    cur ^= 1;
  }
  for (int l = 0; l < A.n_layers; ++l)
    for (int j = tid; j < A.n_rec; j += kFwdThreads)
      A.L[l].z[(size_t)b * A.n_rec + j] = zc[(l * 2 + cur) * npad + j];
  if (tid == 0) {
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
// One thread owns 4 consecutive postsynaptic neurons j0..j0+3 of IT
// consecutive presynaptic rows i0..i0+IT-1 and walks the batch.  For each
// (b, i, j) it reads the traces once, advances them through the block's
// steps, and writes them once.  Per step:
//   e    = psi_j (zbar_i - beta_j epsa)          (dz_j/dW_ji)
//   ebar = kappa ebar + e                        (readout filter on the trace)
//   acc += L_j ebar                              (fp64)
//   epsa = psi_j zbar_i + (rho - beta_j psi_j) epsa   (adaptive j only)
// zbar_i of a (b, i, t) is the same for the whole block: a scalar load.  Trace
// rows are j-contiguous, so a wave moves 1 KiB per 16-byte lane access; the
// next batch element's traces are loaded before the current ones are stored.
template <int IT, bool FIRST>
__global__ __launch_bounds__(256) void trace_kernel(TraceArgs a) {
  const int j0 = (blockIdx.y * blockDim.x + threadIdx.x) * 4;
  const int i0 = blockIdx.x * IT;
  if (j0 >= a.n_post) return;
  const int nit = min(IT, a.n_pre - i0);
  const bool adapt = j0 < a.n_adaptive;
  float bj[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) bj[r] = (j0 + r < a.n_adaptive) ? a.beta : 0.0f;

  double acc[IT][4];
#pragma unroll
  for (int ii = 0; ii < IT; ++ii)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      acc[ii][r] = (FIRST || ii >= nit) ? 0.0 : a.acc[(size_t)(i0 + ii) * a.ldj + j0 + r];

  const size_t bs_e = (size_t)a.n_pre * a.ldj;
  const size_t bs_a = (size_t)a.n_pre * a.lda;
  const size_t zrow = (size_t)a.B * a.Kmax;
  float* pe0 = a.ebar + (size_t)i0 * a.ldj + j0;
  float* pa0 = a.epsa + (size_t)i0 * a.lda + j0;
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};

  f32x4 E[IT], Aa[IT];
#pragma unroll
  for (int ii = 0; ii < IT; ++ii) {
    E[ii] = zero;
    Aa[ii] = zero;
    if (!FIRST && ii < nit) {
      E[ii] = load_nt(pe0 + (size_t)ii * a.ldj);
      if (adapt) Aa[ii] = load_nt(pa0 + (size_t)ii * a.lda);
    }
  }
  for (int b = 0; b < a.B; ++b) {
    f32x4 En[IT], An[IT];
#pragma unroll
    for (int ii = 0; ii < IT; ++ii) {
      En[ii] = zero;
      An[ii] = zero;
      if (!FIRST && b + 1 < a.B && ii < nit) {
        En[ii] = load_nt(pe0 + (size_t)(b + 1) * bs_e + (size_t)ii * a.ldj);
        if (adapt) An[ii] = load_nt(pa0 + (size_t)(b + 1) * bs_a + (size_t)ii * a.lda);
      }
    }
    const float* zk = a.zbarK + ((size_t)i0 * a.B + b) * a.Kmax;
    const float* pp = a.psiK + (size_t)b * a.Kmax * a.ldj + j0;
    const float* lp = a.LK + (size_t)b * a.Kmax * a.ldj + j0;
    for (int t = 0; t < a.steps; ++t) {
      const f32x4 ps = *(const f32x4*)(pp + (size_t)t * a.ldj);
      const f32x4 lv = *(const f32x4*)(lp + (size_t)t * a.ldj);
      double ld[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) ld[r] = (double)lv[r];
      if (adapt) {
        float rb[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) rb[r] = a.rho - bj[r] * ps[r];
#pragma unroll
        for (int ii = 0; ii < IT; ++ii) {
          if (ii < nit) {
            const float zb = zk[(size_t)ii * zrow + t];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float et = ps[r] * (zb - bj[r] * Aa[ii][r]);
              E[ii][r] = fmaf(a.kappa, E[ii][r], et);
              Aa[ii][r] = fmaf(rb[r], Aa[ii][r], ps[r] * zb);
              acc[ii][r] = fma(ld[r], (double)E[ii][r], acc[ii][r]);
            }
          }
        }
      } else {
#pragma unroll
        for (int ii = 0; ii < IT; ++ii) {
          if (ii < nit) {
            const float zb = zk[(size_t)ii * zrow + t];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              E[ii][r] = fmaf(a.kappa, E[ii][r], ps[r] * zb);
              acc[ii][r] = fma(ld[r], (double)E[ii][r], acc[ii][r]);
            }
          }
        }
      }
    }
#pragma unroll
    for (int ii = 0; ii < IT; ++ii) {
      if (ii < nit) {
        store_nt(pe0 + (size_t)b * bs_e + (size_t)ii * a.ldj, E[ii]);
        if (adapt) store_nt(pa0 + (size_t)b * bs_a + (size_t)ii * a.lda, Aa[ii]);
      }
      E[ii] = En[ii];
      Aa[ii] = An[ii];
    }
  }
#pragma unroll
  for (int ii = 0; ii < IT; ++ii)
    if (ii < nit)
#pragma unroll
      for (int r = 0; r < 4; ++r) a.acc[(size_t)(i0 + ii) * a.ldj + j0 + r] = acc[ii][r];
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
hipError_t launch_forward(const FwdArgs& a, hipStream_t s) {
  forward_kernel<<<a.B, kFwdThreads, a.smem, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_gemm_nt(const GemmArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.N, 128), cdiv(a.M, 32), a.splits);
  gemm_nt_kernel<<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_accumulate(const float* part, int splits, size_t split_stride, int M, int N,
                             double* acc, int ld_acc, int first, hipStream_t s) {
  accumulate_kernel<<<cdiv((long long)M * N, 256), 256, 0, s>>>(part, splits, split_stride, M, N,
                                                               acc, ld_acc, first);
  return hipGetLastError();
}

hipError_t launch_trace(const TraceArgs& a, hipStream_t s) {
  constexpr int IT = 4;
  dim3 grid(cdiv(a.n_pre, IT), cdiv(a.n_post, 1024));
  if (a.first)
    trace_kernel<IT, true><<<grid, 256, 0, s>>>(a);
  else
    trace_kernel<IT, false><<<grid, 256, 0, s>>>(a);
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
