// Internal launch interface between the host library (eprop.hip) and the
// gfx950 kernels (kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace eprop {

// Presynaptic vector p^t = [in^t ; z^{t-1}] as fp32 rows of P (the A operand of
// the drive GEMM) and its alpha filter zbarT[i][b] = alpha*zbarT[i][b] + p.
struct PresynArgs {
  const uint8_t* in;   // [B][n_inl]
  const uint8_t* zprev;  // [B][n_rec]
  float* P;            // [>=B][ldp]
  float* zbarT;        // [n_pre][ldz]
  int B, n_inl, n_rec, n_pre, ldp, ldz;
  float alpha;
};
hipError_t launch_presyn(const PresynArgs& a, hipStream_t s);

// C_part[s][m][n] = sum_{k in split s} A[m][k] * Bm[n][k]   (fp32 MFMA).
// A has >= round_up(M,32) rows, Bm >= round_up(N,32) rows, both zero padded
// to K columns (K a multiple of 16).  Split s covers [s*k_chunk, min(K,(s+1)*k_chunk)).
struct GemmArgs {
  const float* A;
  const float* Bm;
  float* C;
  int M, N, K, lda, ldb, ldc;
  int splits, k_chunk;
  size_t split_stride;  // elements between consecutive split outputs
};
hipError_t launch_gemm_nt(const GemmArgs& a, hipStream_t s);

// Neuron step (Eq. 8 with reset and adaptive threshold) and surrogate.
struct NeuronArgs {
  const float* Ipart; int splits; size_t split_stride; int ldI;
  float* v; float* a;          // [B][n_rec]
  const uint8_t* zprev; uint8_t* zcur;   // [B][n_rec]
  float* Zf; int ldzf;         // fp32 spikes, A operand of the readout GEMM
  float* psi; int ldj;         // [B][ldj]
  uint32_t* spikes; int W32;   // optional [B][W32]
  int B, n_rec, n_adaptive;
  float alpha, rho, thr, beta, gamma_over_thr;
};
hipError_t launch_neuron(const NeuronArgs& a, hipStream_t s);

// Leaky readout, softmax cross-entropy, learning signal L = W_out^T delta,
// kappa-filtered spikes.
struct ReadoutArgs {
  const float* Ypart; int splits; size_t split_stride; int ldY;
  float* y; float* delta;      // [B][K]
  const int32_t* labels;
  const float* Wout; int ldo;  // packed [K][ldo]
  const uint8_t* zcur;         // [B][n_rec]
  float* L; float* ztil; int ldj;   // [B][ldj]
  double* lossacc;             // [B]
  int* err_flag;
  int B, K, n_rec;
  float kappa;
};
hipError_t launch_readout(const ReadoutArgs& a, hipStream_t s);

// dW_out[k][j] += sum_b delta[b][k] * ztil[b][j]   (fp64 accumulator).
struct DwoutArgs {
  const float* delta; const float* ztil; int ldj;
  double* accout; int ld_acc;
  int B, K, n_rec, first;
};
hipError_t launch_dwout(const DwoutArgs& a, hipStream_t s);

// Eligibility vectors and gradient accumulation, one pass over the traces.
struct TraceArgs {
  float* ebar;     // [B][n_pre][ldj]
  float* epsa;     // [B][n_pre][lda]
  double* acc;     // [n_pre][ldj]
  const float* zbarT; int ldz;   // [n_pre][ldz]
  const float* psi; const float* L;   // [B][ldj]
  int B, n_pre, n_post, ldj, n_adaptive, lda;
  float kappa, rho, beta;
  int first;       // 1: previous traces and accumulators are zero (not read)
};
hipError_t launch_trace(const TraceArgs& a, hipStream_t s);

// Gradient read-out: dW[j][i] = acc[i][j] (recurrent diagonal zeroed),
// dWout[k][j] = accout[k][j], loss = sum_b lossacc[b]; valid = 0 writes zeros.
struct GradsArgs {
  const double* acc; int ldj; float* dW; int n_pre, n_post, n_inl, recurrent;
  const double* accout; int ld_acc; float* dWout; int K;
  int valid;
};
hipError_t launch_grads(const GradsArgs& a, hipStream_t s);
hipError_t launch_loss(const double* lossacc, int B, int n_layers, size_t layer_stride,
                       double* out, hipStream_t s);

// W [rows][cols] (row-major, ld = cols) -> dst [>=rows][ldd], zero padded.
hipError_t launch_pack(const float* src, int rows, int cols, float* dst, int ldd, int rows_pad,
                       hipStream_t s);

}  // namespace eprop
