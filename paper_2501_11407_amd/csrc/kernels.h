// Internal launch interface between the host library (eprop.hip) and the
// gfx950 kernels (kernels.hip).  Not part of the public ABI.
//
// The sequence is processed in blocks of up to Kmax timesteps.  For a block,
// the forward kernel runs the network for every step (one workgroup per
// batch element) and leaves per-step vectors in "K buffers" (row r = t*Bp + b):
//   psiK   [Kmax*Bp][ldv]  pseudo-derivative (ldv = n_rec rounded to 256)
//   deltaK [rows][ldk]     readout error (softmax - onehot)
//   ztK    [rows][ldn]     kappa-filtered spikes
//   zbarK  [B][Kmax][ldi]  filtered presynaptic vector
// Two MFMA GEMMs follow: the learning signal LK = deltaK * W_out (rows as
// psiK) and the readout gradient dW_out += deltaK^T * ztK.  The eligibility
// kernel then advances every synapse's traces through the block's steps with
// one read and one write of the traces.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace eprop {

constexpr int kFwdThreads = 1024;              // forward workgroup: one batch element
constexpr int kFwdWaves = kFwdThreads / 64;
constexpr int kFwdXSteps = 8;                  // input spikes staged in shared memory per load
constexpr int kTraceWaves = 4;         // waves per eligibility workgroup (same 256 neurons)
constexpr int kTraceChunk = 8;         // steps staged in shared memory at a time
constexpr int kRowPad = 16;            // n_pre padded to a multiple of this (row group)

struct FwdLayer {
  const float* Wt; int ldw;      // transposed drive weights [n_pre][ldw]
  const float* WoutT;            // transposed readout weights [n_rec_pad][ldk]
  float* v; float* a; float* ztil;   // state [B][n_rec]
  uint8_t* z;                    // state: spikes of the last step [B][n_rec]
  float* zbar;                   // state [B][n_pre]
  float* y;                      // state [B][K_out]
  double* lossacc;               // [B]
  float* psiK;                   // [rows][ldj]
  float* zbarK;                  // [B][Kmax][ldi]
  float* deltaK; float* ztK;     // [rows][ldk], [rows][ldn]
  int n_inl, n_pre, rows_per_wave, ldi;
};

struct FwdArgs {
  FwdLayer L[2];
  int n_layers;
  const uint8_t* x;              // [steps][B][n_in]
  int n_in;
  const int32_t* labels;
  int* err_flag;
  uint32_t* spikes;              // NULL or [steps][n_layers][B][W32]
  int W32;
  int B, Bp, n_rec, K_out, n_adaptive, Kmax, steps, ldj, ldk, ldn, jlist;  // ldj: row stride of psiK
  float alpha, rho, kappa, thr, beta, gamma_over_thr;
  size_t smem;
};
hipError_t launch_forward(const FwdArgs& a, hipStream_t s);

// NT: C_part[s][m][n] = sum_{k in split s} A[m][k] * Bm[n][k]
// TN: C_part[s][m][n] = sum_{k in split s} A[k][m] * Bm[k][n]
// fp32 MFMA.  Operands are zero padded: A and Bm provide round_up(M,32) and
// round_up(N,32) rows (NT) or columns (TN), and K is a multiple of 16.
// Split s covers k in [s*k_chunk, min(K,(s+1)*k_chunk)).
struct GemmArgs {
  const float* A;
  const float* Bm;
  float* C;
  int M, N, K, lda, ldb, ldc;
  int splits, k_chunk;
  size_t split_stride;  // elements between consecutive split outputs
};
hipError_t launch_gemm_nt(const GemmArgs& a, hipStream_t s);
hipError_t launch_gemm_tn(const GemmArgs& a, hipStream_t s);

// acc[m][n] (fp64, row stride ld_acc) = (first ? 0 : acc) + sum_s part[s][m][n].
hipError_t launch_accumulate(const float* part, int splits, size_t split_stride, int M, int N,
                             double* acc, int ld_acc, int first, hipStream_t s);

// Eligibility vectors and gradient accumulation over `steps` timesteps.
struct TraceArgs {
  float* ebar;     // [B][n_pre_pad][ldj]
  float* epsa;     // [B][n_pre_pad][lda]
  double* acc;     // [n_pre_pad][ldj]
  const float* zbarK;                 // [B][Kmax][ldi]
  const float* psiK; const float* LK; // [rows][ldv], row t*Bp + b, ldv a multiple of 256
  int B, Bp, n_pre_pad, n_post, ldj, ldv, n_adaptive, lda, Kmax, ldi, steps;
  int n_seg_a, n_seg_l;   // 256-neuron segments holding adaptive neurons, and the rest
  float kappa, rho, beta;
  int first;       // 1: traces and accumulators start at zero (not read)
};
hipError_t launch_trace(const TraceArgs& a, hipStream_t s);

// Gradient read-out: dW[j][i] = acc[i][j] (recurrent diagonal zeroed),
// dWout[k][j] = accout[k][j]; valid = 0 writes zeros.
struct GradsArgs {
  const double* acc; int ldj; float* dW; int n_pre, n_post, n_inl, recurrent;
  const double* accout; int ld_acc; float* dWout; int K;
  int valid;
};
hipError_t launch_grads(const GradsArgs& a, hipStream_t s);
hipError_t launch_loss(const double* lossacc, int B, int n_layers, size_t layer_stride,
                       double* out, hipStream_t s);

// src [rows][cols] row-major -> dst [dst_rows][ldd] (transpose = 0) or
// dst[c][r] = src[r][c] (transpose = 1); every other element of dst is zero.
hipError_t launch_pack(const float* src, int rows, int cols, float* dst, int ldd, int dst_rows,
                       int transpose, hipStream_t s);

}  // namespace eprop
