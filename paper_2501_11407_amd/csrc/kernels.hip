// gfx950 kernels of the online e-prop step.
//
// Built with -ffp-contract=off: every a*b+c written below is a rounded
// multiply followed by a rounded add unless fmaf/fma is spelled out.  The
// neuron step relies on this to reproduce fp32 spike decisions operation by
// operation; the trace and accumulation kernels use explicit fused
// multiply-adds where precision only gains from them.
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

inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

// ---------------------------------------------------------------- presynaptic
// One thread per (i, b), b fastest so the zbarT row update is coalesced.
__global__ __launch_bounds__(256) void presyn_kernel(PresynArgs a) {
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)a.n_pre * a.B) return;
  const int b = (int)(idx % a.B);
  const int i = (int)(idx / a.B);
  const uint8_t s = (i < a.n_inl) ? a.in[(size_t)b * a.n_inl + i]
                                  : a.zprev[(size_t)b * a.n_rec + (i - a.n_inl)];
  const float p = s ? 1.0f : 0.0f;
  a.P[(size_t)b * a.ldp + i] = p;
  float* zb = a.zbarT + (size_t)i * a.ldz + b;
  *zb = a.alpha * *zb + p;
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

// ---------------------------------------------------------------- neuron step
// One thread per (b, j).  Operation order, one rounding each:
//   v = alpha*v; v = v + I; v = v - thr*z_prev
//   a = rho*a;   a = a + z_prev
//   A = beta_j*a; A = thr + A;  x = v - A;  z = x > 0
//   psi = (gamma/thr) * max(0, 1 - |x|/thr)
__global__ __launch_bounds__(256) void neuron_kernel(NeuronArgs a) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const int b = blockIdx.y;
  bool z = false;
  if (j < a.n_rec) {
    float I = 0.0f;
    for (int s = 0; s < a.splits; ++s) I += a.Ipart[s * a.split_stride + (size_t)b * a.ldI + j];
    const size_t o = (size_t)b * a.n_rec + j;
    const float zp = a.zprev[o] ? 1.0f : 0.0f;
    float v = a.alpha * a.v[o];
    v = v + I;
    v = v - a.thr * zp;
    float ad = a.rho * a.a[o];
    ad = ad + zp;
    const float bj = (j < a.n_adaptive) ? a.beta : 0.0f;
    float A = bj * ad;
    A = a.thr + A;
    const float x = v - A;
    a.v[o] = v;
    a.a[o] = ad;
    z = x > 0.0f;
    a.zcur[o] = z ? 1 : 0;
    a.Zf[(size_t)b * a.ldzf + j] = z ? 1.0f : 0.0f;
    const float u = 1.0f - fabsf(x) / a.thr;
    a.psi[(size_t)b * a.ldj + j] = a.gamma_over_thr * fmaxf(u, 0.0f);
  }
  if (a.spikes) {
    const unsigned long long m = __ballot(z);
    const int lane = threadIdx.x & 63;
    const int w0 = (j - lane) >> 5;   // first 32-bit word of this wave's 64 neurons
    uint32_t* row = a.spikes + (size_t)b * a.W32;
    if (lane == 0 && w0 < a.W32) row[w0] = (uint32_t)m;
    if (lane == 1 && w0 + 1 < a.W32) row[w0 + 1] = (uint32_t)(m >> 32);
  }
}

// ---------------------------------------------------------------- readout
// One block per batch element.  Shared memory: y[K], delta[K].
__global__ __launch_bounds__(256) void readout_kernel(ReadoutArgs a) {
  extern __shared__ float sm[];
  float* sy = sm;
  float* sd = sm + a.K;
  __shared__ float s_max, s_sum;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int label = a.labels[b];
  const bool label_ok = label >= 0 && label < a.K;

  for (int k = tid; k < a.K; k += blockDim.x) {
    float Y = 0.0f;
    for (int s = 0; s < a.splits; ++s) Y += a.Ypart[s * a.split_stride + (size_t)b * a.ldY + k];
    float y = a.kappa * a.y[(size_t)b * a.K + k];
    y = y + Y;
    a.y[(size_t)b * a.K + k] = y;
    sy[k] = y;
  }
  __syncthreads();
  if (tid < kWave) {
    float m = -INFINITY;
    for (int k = tid; k < a.K; k += kWave) m = fmaxf(m, sy[k]);
    m = wave_max(m);
    float se = 0.0f;
    for (int k = tid; k < a.K; k += kWave) se += expf(sy[k] - m);
    se = wave_sum(se);
    if (tid == 0) {
      s_max = m;
      s_sum = se;
      if (label_ok) {
        a.lossacc[b] += log((double)se) - ((double)sy[label] - (double)m);
      } else {
        *a.err_flag = 1;
      }
    }
  }
  __syncthreads();
  const float m = s_max, se = s_sum;
  for (int k = tid; k < a.K; k += blockDim.x) {
    const float d = expf(sy[k] - m) / se - ((k == label) ? 1.0f : 0.0f);
    sd[k] = d;
    a.delta[(size_t)b * a.K + k] = d;
  }
  __syncthreads();
  for (int j = tid; j < a.n_rec; j += blockDim.x) {
    float Lj = 0.0f;
    for (int k = 0; k < a.K; ++k) Lj = fmaf(a.Wout[(size_t)k * a.ldo + j], sd[k], Lj);
    a.L[(size_t)b * a.ldj + j] = Lj;
    const float zt = a.zcur[(size_t)b * a.n_rec + j] ? 1.0f : 0.0f;
    float* zt_p = a.ztil + (size_t)b * a.ldj + j;
    *zt_p = a.kappa * *zt_p + zt;
  }
}

// ---------------------------------------------------------------- readout gradient
__global__ __launch_bounds__(256) void dwout_kernel(DwoutArgs a) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const int k = blockIdx.y;
  if (j >= a.n_rec) return;
  double* p = a.accout + (size_t)k * a.ld_acc + j;
  double s = a.first ? 0.0 : *p;
  for (int b = 0; b < a.B; ++b)
    s = fma((double)a.delta[(size_t)b * a.K + k], (double)a.ztil[(size_t)b * a.ldj + j], s);
  *p = s;
}

// ---------------------------------------------------------------- eligibility
// One thread owns 4 consecutive postsynaptic neurons j0..j0+3 of IT
// consecutive presynaptic rows i0..i0+IT-1 and walks the batch.  For each
// (b, i, j):
//   e    = psi_j (zbar_i - beta_j epsa)          (dz_j/dW_ji)
//   ebar = kappa ebar + e                        (readout filter on the trace)
//   acc += L_j ebar                              (fp64)
//   epsa = psi_j zbar_i + (rho - beta_j psi_j) epsa   (adaptive j only)
// zbar_i of a (b, i) is the same for the whole block: a scalar load.  Trace
// rows are j-contiguous, so a wave moves 1 KiB per 16-byte lane access.
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
  float* pe0 = a.ebar + (size_t)i0 * a.ldj + j0;
  float* pa0 = a.epsa + (size_t)i0 * a.lda + j0;
  const float* zb0 = a.zbarT + (size_t)i0 * a.ldz;

  for (int b = 0; b < a.B; ++b) {
    const f32x4 ps = *(const f32x4*)(a.psi + (size_t)b * a.ldj + j0);
    const f32x4 lv = *(const f32x4*)(a.L + (size_t)b * a.ldj + j0);
    float rb[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) rb[r] = a.rho - bj[r] * ps[r];
#pragma unroll
    for (int ii = 0; ii < IT; ++ii) {
      if (ii < nit) {
        const float zb = zb0[(size_t)ii * a.ldz + b];
        f32x4* pe = (f32x4*)(pe0 + (size_t)b * bs_e + (size_t)ii * a.ldj);
        f32x4 e = FIRST ? f32x4{0.f, 0.f, 0.f, 0.f} : *pe;
        if (adapt) {
          f32x4* pa = (f32x4*)(pa0 + (size_t)b * bs_a + (size_t)ii * a.lda);
          f32x4 ea = FIRST ? f32x4{0.f, 0.f, 0.f, 0.f} : *pa;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float et = ps[r] * (zb - bj[r] * ea[r]);
            e[r] = fmaf(a.kappa, e[r], et);
            ea[r] = fmaf(rb[r], ea[r], ps[r] * zb);
          }
          *pa = ea;
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) e[r] = fmaf(a.kappa, e[r], ps[r] * zb);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[ii][r] = fma((double)lv[r], (double)e[r], acc[ii][r]);
        *pe = e;
      }
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
                                                   int ldd, int rows_pad) {
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)rows_pad * ldd) return;
  const int r = (int)(idx / ldd), c = (int)(idx % ldd);
  dst[idx] = (r < rows && c < cols) ? src[(size_t)r * cols + c] : 0.0f;
}

}  // namespace

// ---------------------------------------------------------------- launchers
hipError_t launch_presyn(const PresynArgs& a, hipStream_t s) {
  const long long n = (long long)a.n_pre * a.B;
  presyn_kernel<<<cdiv(n, 256), 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_gemm_nt(const GemmArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.N, 128), cdiv(a.M, 32), a.splits);
  gemm_nt_kernel<<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_neuron(const NeuronArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.n_rec, 256), a.B);
  neuron_kernel<<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_readout(const ReadoutArgs& a, hipStream_t s) {
  readout_kernel<<<a.B, 256, 2 * a.K * sizeof(float), s>>>(a);
  return hipGetLastError();
}

hipError_t launch_dwout(const DwoutArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.n_rec, 256), a.K);
  dwout_kernel<<<grid, 256, 0, s>>>(a);
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

hipError_t launch_pack(const float* src, int rows, int cols, float* dst, int ldd, int rows_pad,
                       hipStream_t s) {
  const long long n = (long long)rows_pad * ldd;
  pack_kernel<<<cdiv(n, 256), 256, 0, s>>>(src, rows, cols, dst, ldd, rows_pad);
  return hipGetLastError();
}

}  // namespace eprop
