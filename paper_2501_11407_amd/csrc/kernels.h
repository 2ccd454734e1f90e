// Internal launch interface between the host library (eprop.hip) and the
// gfx950 kernels (kernels.hip).  Not part of the public ABI.
//
// The sequence is processed in blocks of up to Kmax timesteps.  For a block,
// the forward kernel runs the network for every step (one workgroup per
// batch element) and leaves per-step vectors in "K buffers" (row r = t*Bp + b):
//   psiK   [Kmax*Bp][ldv]  pseudo-derivative (ldv = n_rec rounded to 256)
//   deltaK [rows][ldk]     readout error (softmax - onehot)
//   ztK    [rows][ldn]     kappa-filtered spikes
//   pbits  [B][Kmax/16][ldi]     binary presynaptic vector: per 16-step
//                                chunk and row, one 16-bit word (bit s: step
//                                16 c + s)
//   zstart [B][ldi]              presynaptic filter at the block's start
// Two MFMA GEMMs follow: the learning signal LK = deltaK * W_out (rows as
// psiK) and the readout gradient dW_out += deltaK^T * ztK; then the block
// coefficients of the eligibility recursion and the eligibility kernel, which
// advances every synapse's traces through the block's steps with one read and
// one write of the traces.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace eprop {

constexpr int kFwdThreads = 512;               // forward workgroup: one batch element
constexpr int kFwdWaves = kFwdThreads / 64;
constexpr int kBlockSteps = 512;       // timesteps per block (Kmax)
constexpr int kTileI = 256;            // eligibility workgroup tile: 256 (i) x 16 (j)
constexpr int kTileJ = 16;
constexpr int kRowPad = kTileI;        // n_pre padded to the tile height (ldi)
constexpr int kColPad = kTileJ;        // n_rec padded to the tile width (ldc)

// Forward thread 64 w + l (wave w, lane l) holds the QN neurons
// 64 QN w + 64 q + l, q < QN (QN: neurons per thread, a power of two); the
// int16 drive weights and the input drive store neuron j at position
// tid QN + q of a row of 512 QN, so that a thread reads its QN in one load.
__host__ __device__ inline int fwd_position(int j, int qn) {
  const int w = j / (64 * qn), q = (j / 64) % qn, l = j % 64;
  return (64 * w + l) * qn + q;
}

struct FwdLayer {
  const float* Wt; int ldw;      // transposed drive weights [n_pre][ldw], ldw = 512 QN
  // the same times 2^14 as int16 [n_pre][512 QN] at forward positions; used
  // when *FwdArgs::w16ok (see launch_pack16)
  const int16_t* W16;
  const float* WoutT;            // transposed readout weights [n_rec_pad][ldk]
  float* v; float* a; float* ztil;   // state [B][n_rec]
  uint8_t* z;                    // state: spikes of the last step [B][n_rec]
  float* zbar;                   // state [B][n_pre]
  float* y;                      // state [B][K_out]
  double* lossacc;               // [B]
  float* psiK;                   // [rows][ldj]
  uint16_t* pbits;               // [B][Kmax/16][ldi]
  float* zstart;                 // [B][ldi]
  float* deltaK; float* ztK;     // [rows][ldk], [rows][ldn]
  int n_inl, n_pre, ldi;
};

// The forward handles the p bits, filter and zstart of the recurrent rows
// (and of every row of a second layer); the first layer's input rows, and
// the input part of its drive, come from the input kernels below.
struct FwdArgs {
  FwdLayer L[2];
  int n_layers;
  const float* Iin;              // first layer's input drive [steps][B][512 QN] (launch_input_drive)
  const int* nin;                // [steps][B]: its number of active inputs
  const int32_t* labels;
  int* err_flag;
  uint32_t* spikes;              // NULL or [steps][n_layers][B][W32]
  int W32;
  int B, Bp, n_rec, K_out, n_adaptive, Kmax, steps, ldj, ldk, ldn, jlist;  // ldj: row stride of psiK
  float alpha, rho, kappa, thr, beta, gamma_over_thr;
  float inv_thr;                 // 1/thr (exact for a power-of-two threshold)
  // neuron_model 1: h = A h_prev + b I + r z_prev, spike argument
  // u = c . h - thr (the two-compartment neuron, coefficients derived on the
  // host; v holds h0, a holds h1)
  int model;
  float mA[2][2], mb[2], mr[2], mc[2];
  const int* w16ok;              // [0]: every layer's W16 is exact, [1]: their largest |k|
  // 1: a ninth (service) wave stages the input drive in shared memory (a
  // ring of three steps, 6 KiB per neuron per thread, at the start of smem);
  // required for QN <= 2, allowed for QN == 4, not for more
  int svc;
  size_t smem;
};
hipError_t launch_forward(const FwdArgs& a, hipStream_t s);

// The first layer's input rows over a block of `steps` steps, x [steps][B][n_in]:
// launch_input_drive writes Iin[t][b][512 qn] (forward positions), the sum of
// the drive weights over the step's active inputs in ascending order in fp32
// from 0 (rows from W16 when *w16ok, else Wt), and nin[t][b], their number;
// launch_input_filter advances zbar [B][n_pre] of the input rows over the
// steps (their value at the start into zstart [B][ldi]) and writes their p
// bits into pbits as the forward does for its rows.
struct InputArgs {
  const uint8_t* x; int n_in, B, steps;
  const float* Wt; int ldw; const int16_t* W16; int qn; const int* w16ok;
  float* Iin; int* nin;
  float* zbar; int n_pre; float* zstart; uint16_t* pbits; int ldi; float alpha;
};
hipError_t launch_input_drive(const InputArgs& a, hipStream_t s);
hipError_t launch_input_filter(const InputArgs& a, hipStream_t s);

// NT: C_part[s][m][n] = sum_{k in split s} A[m][k] * Bm[n][k]
// TN: C_part[s][m][n] = sum_{k in split s} A[k][m] * Bm[k][n]
// fp32 MFMA.  Operands are zero padded: A and Bm provide round_up(M,32) and
// round_up(N,32) rows (NT) or columns (TN; the TN kernel reads A only up to
// round_up(M,16) columns), and K is a multiple of 16.
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

// The operands of the eligibility contractions are stored as scaled fp16
// pairs: a value x (times a power-of-two scale 2^e) is hi = fp16(x 2^e) plus
// lo = fp16(x 2^e - hi), together about 22 significant bits.  Per 16-step
// chunk and row, 64 bytes: per quad of steps a 16-byte unit of the four hi
// halves and then the four lo halves.
// The presynaptic operand is binary (bits, expanded to fp16 in the kernel).
constexpr int kChunk = 16;                     // steps per chunk
constexpr int kKC = kBlockSteps / kChunk;      // chunks per block
constexpr int kScalarPlanes = 8;               // see coef_kernel

// Coefficient operands, tile-major: per batch element and chunk, the column
// tiles of kTileJ columns in order, and per tile its operands one after the
// other (U, H, then V in tiles holding adaptive neurons, then W with the
// reset path kept), each 16 rows (the tile's columns) of 16 pair words (the
// chunk's steps), 1 KiB.  The tiles holding adaptive neurons come first.
// One eligibility workgroup's operands of a chunk are one contiguous run.
struct OpLayout {
  int n_jt_a;        // tiles holding adaptive neurons
  int nxa, nxl;      // operands per tile with and without adaptive neurons
  int cw;            // words per chunk: 256 (n_jt_a nxa + (n_jt - n_jt_a) nxl)
  // first word of tile jt within a chunk
  __host__ __device__ int tile(int jt) const {
    return 256 * (jt < n_jt_a ? jt * nxa : n_jt_a * nxa + (jt - n_jt_a) * nxl);
  }
};

// Block coefficients of the eligibility recursion, one thread per (b, j):
// U', V', H' (against the binary presynaptic vector) as scaled fp16 pair
// words in O [B][kKC][ol.cw] (OpLayout; zero for steps <= s < kpad; V' in
// the tiles holding adaptive neurons only), each row with its own
// power-of-two scale, and S [kScalarPlanes][B][ldc] (see coef_kernel).  With
// reset_through the rows are those of the
// recursion with the reset path kept (U = C_E, H = C_g, V = C_A, and W = C_V
// for every j) and S has kScalarPlanesRT planes (see coef_rt_kernel).
constexpr int kScalarPlanesRT = 16;
struct CoefArgs {
  const float* psiK; const float* LK; int ldv, Bp;   // [t*Bp + b][ldv]
  uint32_t* O; OpLayout ol; float* S;
  int B, n_post, n_adaptive, steps, kpad, ldc;
  float kappa, rho, beta, alpha, thr;
  int reset_through;
  // model 1: the generic adjoint pass (coef_gen_kernel) of a step with
  // H_I = A + psi_prev r c^T, F = b p, e = psi c . eps
  int model;
  float gA[2][2], gb[2], gr[2], gc[2];
};
hipError_t launch_coef(const CoefArgs& a, hipStream_t s);


// The traces are stored tile by tile: for batch element b and 256 x 16 tile
// (it, jt), 16 KiB holding the four 64 x 16 wave sub-tiles, each as four
// 16 x 16 blocks bi of 64 lanes x 4 floats, in the order the kernel's lanes
// hold them (see trace_kernel).  epsa covers the n_jt_a tiles that hold
// adaptive neurons.
struct TraceArgs {
  float* ebar;     // [B][n_pre_pad / 256][n_jt][256 * 16]
  float* epsa;     // [B][n_pre_pad / 256][n_jt_a][256 * 16]
  float* epsv;     // reset_through: [B][n_pre_pad / 256][n_jt][256 * 16]
  double* acc;     // [n_split][n_pre_pad][ldj] (row-major)
  size_t acc_stride;
  const uint16_t* pbits;              // [B][kKC][ldi], ldi = n_pre_pad
  const float* zstart;                // [B][ldi] (reset-stopped form only)
  const uint32_t* O; OpLayout ol;     // as CoefArgs
  const float* S;                     // as CoefArgs
  int B, n_pre, n_pre_pad, n_post, ldj, n_adaptive, ldi, ldc, kpad, n_split;
  int n_jt, n_jt_a;   // tiles along j: all, and those holding adaptive neurons
  float kappa_K;   // kappa^steps
  int first;       // 1: traces and accumulators start at zero (not read)
  int reset_through;   // 1: the recursion with the reset path kept
};
hipError_t launch_trace(const TraceArgs& a, hipStream_t s);

// Gradient read-out: dW[j][i] = sum over splits s of acc[s][i][j] (in split
// order; recurrent diagonal zeroed), dWout[k][j] = accout[k][j]; valid = 0
// writes zeros.
struct GradsArgs {
  const double* acc; int ldj; int n_split; size_t acc_stride;
  float* dW; int n_pre, n_post, n_inl, recurrent;
  const double* accout; int ld_acc; float* dWout; int K;
  int valid;
};
// Every layer's dW and dW_out and (loss not NULL) the loss, in one launch.
struct ReadoutArgs {
  GradsArgs g[2];
  int n_layers;
  const double* lossacc; int B; size_t layer_stride; double* loss;
};
hipError_t launch_readout(const ReadoutArgs& r, hipStream_t s);

// src [rows][cols] row-major -> dst [dst_rows][ldd] (transpose = 0) or
// dst[c][r] = src[r][c] (transpose = 1); every other element of dst is zero.
hipError_t launch_pack(const float* src, int rows, int cols, float* dst, int ldd, int dst_rows,
                       int transpose, hipStream_t s);

// Drive weights W [n_rec][n_pre] (row-major) -> W16 as FwdLayer::W16 for
// QN = the forward's neurons per thread.  ok[0] is cleared unless every
// weight is k 2^-14 with integer |k| <= 32767, and ok[1] becomes the largest
// |k| seen (atomic max).  A drive over at most 2^24 / max|k| active rows then
// has every partial sum an integer of at most 2^24 units in any order, exact
// in fp32, and summing k as integers gives the fp32 sequential sum bit for
// bit; the forward decides this per step.  launch_set_flag sets ok[0] = value
// and ok[1] = 0 before the layers are packed.
hipError_t launch_pack16(const float* W, int n_rec, int n_pre, int16_t* W16, int qn, int* ok,
                         hipStream_t s);
hipError_t launch_set_flag(int* flag, int value, hipStream_t s);
// Zeroes `bytes` bytes at `p` (a fill kernel, not a memset node).
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);
// Up to kMax device ranges zeroed by one launch (ranges of 0 bytes allowed).
struct ZeroRanges {
  static constexpr int kMax = 16;
  void* p[kMax];
  size_t bytes[kMax];
  int n;
};
hipError_t launch_zero_many(const ZeroRanges& r, hipStream_t s);

// Online weight application for one layer: the weights in use become
// W0 - lr * G rounded to the nearest multiple of 2^-14 (ties to even), G the
// gradient accumulated so far (acc summed over its splits in split order,
// accout); the recurrent diagonal keeps W0.  Writes Wt (transposed fp32), W16
// (as launch_pack16, clearing *ok where a weight has no exact int16 form) and
// WoutT [n_rec][ldk].
struct OnlineArgs {
  const float* W0; const float* Wout0;      // the caller's W [n_rec][n_pre], W_out [K][n_rec]
  const double* acc; int ldj, n_split; size_t acc_stride;
  const double* accout; int ld_acc;
  float* Wt; int ldw; int16_t* W16; int qn; int* ok;
  float* WoutT; int ldk;
  int n_rec, n_pre, n_inl, recurrent, K;
  double lr;
};
hipError_t launch_online_update(const OnlineArgs& a, hipStream_t s);
// The weights in use back in the caller's layouts: W [n_rec][n_pre] from Wt,
// W_out [K][n_rec] from WoutT.
hipError_t launch_unpack_weights(const float* Wt, int ldw, const float* WoutT, int ldk, int n_rec,
                                 int n_pre, int K, float* W, float* Wout, hipStream_t s);
// neurons per forward thread for n_rec neurons (a power of two, at most 16)
int forward_qn(int n_rec);

}  // namespace eprop
