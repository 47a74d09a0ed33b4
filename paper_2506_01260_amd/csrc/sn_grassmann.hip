// The subspace update of Sec. 4.5 on the GPU: the off-subspace loss, the
// accumulation behind the Euclidean gradient -2 S U (Sec. 6), and the
// Riemannian step with its QR retraction.
//
// Accumulation.  Sec. 6 accumulates S = (1/K) sum_t G_t^T G_t (d x d) every
// iteration and multiplies by U at the update.  U does not change between two
// updates, so S U = (1/K) sum_t G_t^T (G_t U): the state keeps
// Y = sum_t G_t^T C_t with C_t = G_t U (d x k, float64) instead of S.  Per
// iteration that is a contraction over tokens of 2 N d k flops, bound by
// reading G, instead of the 2 N d^2 flops of G^T G.
//
// Loss.  |G (I - U U^T)|_F^2 = sum over rows g of
//   |g|^2 - 2 |c|^2 + c (U^T U) c^T,  c = g U,
// which is exact for any stored U; with D = U^T U - I (a section of the
// packed basis) the row term is |g|^2 - |c|^2 + c D c^T.
//
// MFMA path (bf16, d a multiple of 64, k <= 128), per accumulate:
//   1. the staged compress kernel with the subspace-update epilogue: per row
//      |g|^2 (summed with the stages), c = g U, and the loss term (c D c^T
//      on the matrix cores), summed per workgroup; C split into bf16 hi + lo
//      in the MFMA operand layout of a contraction over tokens (through
//      LDS); C in bf16 for the wire when asked;
//   2. the weight projection's pass-1 kernel with tokens as the contraction:
//      Tp[split][i][j] = sum over the split's rows of C_hi/lo[n, j] G[n, i];
//   3. finish_kernel: Y += the splits and halves in a fixed order (float64),
//      the loss partials into the state's scalars.
// Generic path (fp32, other shapes): float64 kernels with one thread per
// output, the loss taken directly as sum (g - c U^T)^2.
//
// Step (float64 throughout): Z = U^T Y, A = U + (2 eta / K)(Y - U Z), then
// two rounds of Cholesky QR (Gram matrix, Cholesky factor R with a positive
// diagonal, Q = A R^{-1}): the thin QR with diag(R) > 0, to rounding.
#include "sn_mfma_common.h"

namespace sn {

namespace {

// ---------------------------------------------------------------------------
// plans
// ---------------------------------------------------------------------------
struct AccPlan {
  bool mfma = false;
  int kt = 0;          // C32 row length kp = 16 kt
  int nparts = 0;      // operands of the token contraction: 1 = [C_hi | C_lo], 2 = C_hi, C_lo
  int ktb = 0;         // 16-column tiles per operand
  int ds = 0;          // token splits
  int64_t rows = 0;    // tokens per split, a multiple of 128
  int64_t npad = 0;    // ds * rows >= N
  int64_t m_pad = 0;   // d rounded up to 128
  int64_t nlblk = 0;   // loss partials (at most one per 64 rows on the MFMA path, 256 on the generic)
  size_t off_c = 0, off_frag = 0, off_part = 0, off_tp = 0, total = 0;
};

AccPlan acc_plan(const PackLayout &L, int64_t N, bool mfma) {
  AccPlan P;
  P.mfma = mfma;
  P.nlblk = mfma ? ceil_div(N, 64) : ceil_div(N, 256);
  size_t off = 0;
  if (mfma) {
    P.kt = L.kt;
    if (2 * L.k <= 16 * kMfmaMaxKT) {
      P.nparts = 1;
      P.ktb = static_cast<int>(ceil_div(2 * L.k, 16));
    } else {
      P.nparts = 2;
      P.ktb = L.kt;
    }
    int64_t ds = ceil_div(N, 4096);
    ds = ds < 1 ? 1 : (ds > 8 ? 8 : ds);
    P.rows = ceil_div(ceil_div(N, ds), 128) * 128;
    if (P.rows < 128) P.rows = 128;  // N = 0: the plan is only sized
    P.ds = static_cast<int>(ceil_div(N > 0 ? N : 1, P.rows));
    P.npad = P.ds * P.rows;
    P.m_pad = ceil_div(L.d, 128) * 128;
    P.off_frag = off;
    off = align256(off + static_cast<size_t>(P.nparts) * (P.npad / 32) * P.ktb * 1024);
    P.off_part = off;
    off = align256(off + static_cast<size_t>(P.nlblk) * 8);
    P.off_tp = off;
    off = align256(off + static_cast<size_t>(P.nparts) * P.ds * P.m_pad * 16 * P.ktb * 4);
  } else {
    P.off_c = off;
    off = align256(off + static_cast<size_t>(N) * L.k * 8);
    P.off_part = off;
    off = align256(off + static_cast<size_t>(P.nlblk) * 8);
  }
  P.total = off;
  return P;
}

struct StepPlan {
  int64_t nch = 0, rpc = 0;  // row chunks of the Gram reductions
  size_t off_a = 0, off_q = 0, off_part = 0, off_z = 0, off_gram = 0, off_r = 0,
         off_status = 0, total = 0;
};

StepPlan step_plan(int64_t d, int64_t k) {
  StepPlan P;
  P.nch = ceil_div(d, 32);
  if (P.nch > 256) P.nch = 256;
  P.rpc = ceil_div(d, P.nch);
  P.nch = ceil_div(d, P.rpc);
  const size_t dk = static_cast<size_t>(d) * k * 8, kk = static_cast<size_t>(k) * k * 8;
  size_t off = 0;
  P.off_a = off;
  off = align256(off + dk);
  P.off_q = off;
  off = align256(off + dk);
  P.off_part = off;
  off = align256(off + P.nch * kk);
  P.off_z = off;
  off = align256(off + kk);
  P.off_gram = off;
  off = align256(off + kk);
  P.off_r = off;
  off = align256(off + kk);
  P.off_status = off;
  off = align256(off + 2 * sizeof(int));
  P.total = off;
  return P;
}

__device__ __forceinline__ double *state_y(double *state) {
  return reinterpret_cast<double *>(reinterpret_cast<char *>(state) + kGrassStateHead);
}
__device__ __forceinline__ const double *state_y(const double *state) {
  return reinterpret_cast<const double *>(reinterpret_cast<const char *>(state) +
                                          kGrassStateHead);
}

// fixed-order tree sum of 256 float64 values in LDS; thread 0 gets the total
__device__ __forceinline__ double block_sum256(double v, double *red) {
  red[threadIdx.x] = v;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (static_cast<int>(threadIdx.x) < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  return red[0];
}

// float64 -> bf16, round to nearest even, without double rounding: round to
// float by truncation, make the float odd when that was inexact (round to
// odd keeps the information RNE at 8 bits needs: Boldo and Melquiond,
// "Emulation of FMA and correctly rounded sums: proved algorithms using
// rounding to odd", IEEE Trans. Computers 57(4), 2008), then RNE to bf16.
__device__ __forceinline__ bf16_t bf16_from_f64(double x) {
  float f = __double2float_rz(x);
  if (static_cast<double>(f) != x && x == x) f = __uint_as_float(__float_as_uint(f) | 1u);
  return from_f32<bf16_t>(f);
}

// ---------------------------------------------------------------------------
// state
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void reset_kernel(double *__restrict__ state, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) state[i] = 0.0;
}

// ---------------------------------------------------------------------------
// accumulate, MFMA path
// ---------------------------------------------------------------------------
// ---------------------------------------------------------------------------
// accumulate, generic path (float64, one thread per output)
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void gen_coeff_kernel(const T *__restrict__ G, int64_t ldg,
                                                        const float *__restrict__ U32, int64_t N,
                                                        int64_t d, int64_t k,
                                                        double *__restrict__ C64) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= N * k) return;
  const int64_t n = idx / k, j = idx - (idx / k) * k;
  double acc = 0.0;
  for (int64_t r = 0; r < d; ++r)
    acc += static_cast<double>(to_f32(G[n * ldg + r])) * static_cast<double>(U32[r * k + j]);
  C64[idx] = acc;
}

template <typename T>
__global__ __launch_bounds__(256) void gen_loss_kernel(const T *__restrict__ G, int64_t ldg,
                                                       const float *__restrict__ U32,
                                                       const double *__restrict__ C64, int64_t N,
                                                       int64_t d, int64_t k,
                                                       double *__restrict__ part) {
  __shared__ double red[256];
  const int64_t n = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  double l = 0.0;
  if (n < N) {
    for (int64_t r = 0; r < d; ++r) {
      double v = static_cast<double>(to_f32(G[n * ldg + r]));
      for (int64_t j = 0; j < k; ++j) v -= C64[n * k + j] * static_cast<double>(U32[r * k + j]);
      l += v * v;
    }
  }
  const double tot = block_sum256(l, red);
  if (threadIdx.x == 0) part[blockIdx.x] = tot;
}

template <typename T>
__global__ __launch_bounds__(256) void gen_su_kernel(const T *__restrict__ G, int64_t ldg,
                                                     const double *__restrict__ C64, int64_t N,
                                                     int64_t d, int64_t k,
                                                     double *__restrict__ state) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= d * k) return;
  const int64_t i = idx / k, j = idx - (idx / k) * k;
  double acc = 0.0;
  for (int64_t n = 0; n < N; ++n)
    acc += static_cast<double>(to_f32(G[n * ldg + i])) * C64[n * k + j];
  state_y(state)[idx] += acc;
}

// ---------------------------------------------------------------------------
// accumulate: fold the partial results into the state
// ---------------------------------------------------------------------------
// Y[i, j] += sum over splits s of (T0[s][i][j] + T1[s][i][j']) where the hi
// and lo halves are columns j and k + j of one operand (nparts 1) or column j
// of two (nparts 2).  Thread 0 adds the loss partials and counts the call.
__global__ __launch_bounds__(256) void finish_kernel(const float *__restrict__ tp, int ds,
                                                     int64_t m_pad, int64_t kpb, int nparts,
                                                     int64_t d, int64_t k, int add_tp,
                                                     const double *__restrict__ part,
                                                     int64_t nlblk, int with_su,
                                                     double *__restrict__ state) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (add_tp && idx < d * k) {
    const int64_t i = idx / k, j = idx - (idx / k) * k;
    const int64_t part_stride = static_cast<int64_t>(ds) * m_pad * kpb;
    double acc = 0.0;
    for (int sp = 0; sp < ds; ++sp) {
      const float *row = tp + (sp * m_pad + i) * kpb;
      acc += static_cast<double>(row[j]);
      acc += static_cast<double>(nparts == 1 ? row[k + j] : row[part_stride + j]);
    }
    state_y(state)[idx] += acc;
  }
  if (blockIdx.x != 0) return;
  // block 0: the loss partials, each thread a strided subset in order, then a tree
  __shared__ double red[256];
  double v = 0.0;
  for (int64_t b = threadIdx.x; b < nlblk; b += 256) v += part[b];
  const double sum = block_sum256(v, red);
  if (threadIdx.x == 0) {
    state[0] += sum;
    state[1] += 1.0;
    state[2] = state[0] / state[1];
    if (with_su) state[3] += 1.0;
  }
}

// ---------------------------------------------------------------------------
// step
// ---------------------------------------------------------------------------
// partial[c][a * k + b] = sum over the rows r of chunk c of A[r, a] B[r, b];
// the chunk's rows (at most kGramRows) are staged in LDS as float64.
constexpr int kGramRows = 32;
template <typename TA, typename TB>
__global__ __launch_bounds__(256) void gram_partial_kernel(const TA *__restrict__ A, int64_t lda,
                                                           const TB *__restrict__ B, int64_t ldb,
                                                           int64_t d, int64_t k, int64_t rpc,
                                                           double *__restrict__ partial) {
  __shared__ double sa[kGramRows * kGrassMaxK], sb[kGramRows * kGrassMaxK];
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * rpc;
  const int64_t r1 = r0 + rpc < d ? r0 + rpc : d;
  const int64_t kk = k * k;
  // outputs in groups of 16 per thread (k <= 64: one group)
  for (int64_t og = 0; og < kk; og += 16 * 256) {
    double acc[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = 0.0;
    for (int64_t c0 = r0; c0 < r1; c0 += kGramRows) {
      const int64_t nrow = r1 - c0 < kGramRows ? r1 - c0 : kGramRows;
      __syncthreads();
      for (int64_t e = threadIdx.x; e < nrow * k; e += 256) {
        const int64_t rr = e / k, cc = e - (e / k) * k;
        sa[e] = static_cast<double>(A[(c0 + rr) * lda + cc]);
        sb[e] = static_cast<double>(B[(c0 + rr) * ldb + cc]);
      }
      __syncthreads();
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int64_t o = og + threadIdx.x + 256 * i;
        if (o < kk) {
          const int64_t a = o / k, b = o - (o / k) * k;
          double v = acc[i];
          for (int64_t rr = 0; rr < nrow; ++rr) v += sa[rr * k + a] * sb[rr * k + b];
          acc[i] = v;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int64_t o = og + threadIdx.x + 256 * i;
      if (o < kk) partial[blockIdx.x * kk + o] = acc[i];
    }
  }
}

__global__ __launch_bounds__(256) void gram_reduce_kernel(const double *__restrict__ partial,
                                                          int64_t nch, int64_t kk,
                                                          double *__restrict__ out) {
  const int64_t o = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (o >= kk) return;
  double acc = 0.0;
#pragma unroll 8
  for (int64_t c = 0; c < nch; ++c) acc += partial[c * kk + o];
  out[o] = acc;
}

// A = U + (2 eta / K) (Y - U Z), Z = U^T Y: the step U - eta T against the
// Riemannian gradient T = -(2 / K)(Y - U U^T Y) of the accumulated loss.
__global__ __launch_bounds__(256) void update_kernel(const float *__restrict__ U32,
                                                     const double *__restrict__ state,
                                                     const double *__restrict__ Z, double eta,
                                                     int64_t d, int64_t k, double *__restrict__ A,
                                                     int *__restrict__ status) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx == 0) {
    status[0] = 0;
    status[1] = 0;
  }
  if (idx >= d * k) return;
  const int64_t r = idx / k, b = idx - (idx / k) * k;
  const double ks = state[3];
  const double sc = ks > 0.0 ? 2.0 * eta / ks : 0.0;
  double acc = state_y(state)[idx];
  for (int64_t a = 0; a < k; ++a) acc -= static_cast<double>(U32[r * k + a]) * Z[a * k + b];
  A[idx] = static_cast<double>(U32[idx]) + sc * acc;
}

// Cholesky factor R (upper, positive diagonal) of the k x k Gram matrix,
// gram = R^T R, and its inverse X = R^{-1} (upper), written to Rinv: one
// workgroup, everything in LDS.  A non-positive, NaN or overflowing pivot
// sets *status.
__global__ __launch_bounds__(256) void chol_kernel(const double *__restrict__ gram, int64_t k64,
                                                   double *__restrict__ Rinv,
                                                   int *__restrict__ status) {
  __shared__ double A[kGrassMaxK][kGrassMaxK + 1];
  __shared__ double xd[kGrassMaxK];
  __shared__ int bad;
  const int k = static_cast<int>(k64);
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;  // 16 x 16 thread grid
  for (int i = ty; i < k; i += 16)
    for (int l = tx; l < k; l += 16) A[i][l] = gram[i * k + l];
  if (tid == 0) bad = 0;
  __syncthreads();
  for (int j = 0; j < k; ++j) {
    if (tid == 0) {
      double p = A[j][j];
      if (!(p > 0.0 && p <= 1.0e300)) {  // non-positive, NaN or overflowing pivot
        bad = 1;
        p = 1.0;
      }
      A[j][j] = sqrt(p);
    }
    __syncthreads();
    const double inv = 1.0 / A[j][j];
    for (int l = j + 1 + tid; l < k; l += 256) A[j][l] *= inv;
    __syncthreads();
    for (int i = j + 1 + ty; i < k; i += 16) {
      const double rji = A[j][i];
      for (int l = i + ((tx - i) % 16 + 16) % 16; l < k; l += 16) A[i][l] -= rji * A[j][l];
    }
    __syncthreads();
  }
  // X = R^{-1}: thread b solves R x = e_b by back substitution; x_i (i < b)
  // is kept at A[b][i], below the diagonal (the factor lives on and above
  // it), and x_b in xd[b]
  for (int b = tid; b < k; b += 256) {
    xd[b] = 1.0 / A[b][b];
    for (int i = b - 1; i >= 0; --i) {
      double v = -A[i][b] * xd[b];
      for (int l = i + 1; l < b; ++l) v -= A[i][l] * A[b][l];
      A[b][i] = v / A[i][i];
    }
  }
  __syncthreads();
  for (int i = ty; i < k; i += 16)
    for (int b = tx; b < k; b += 16) Rinv[i * k + b] = i < b ? A[b][i] : (i == b ? xd[b] : 0.0);
  if (tid == 0 && bad) *status = 1;
}

// Q = A R^{-1}, one thread per element: Q[r, b] = sum_{a <= b} A[r, a] X[a, b].
// OUT 0: float64 to the workspace; OUT 1 / 2: the new basis as float32 / bf16
// (rounded once from float64), or the old basis unchanged when either
// Cholesky factorisation failed.
template <int OUT>
__global__ __launch_bounds__(256) void tri_apply_kernel(const double *__restrict__ A,
                                                        const double *__restrict__ Rinv,
                                                        int64_t d, int64_t k,
                                                        const int *__restrict__ status,
                                                        const float *__restrict__ U32, void *out,
                                                        int64_t ldo, int32_t *err_flag) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= d * k) return;
  const int64_t r = idx / k, b = idx - (idx / k) * k;
  double v = 0.0;
  for (int64_t a = 0; a <= b; ++a) v += A[r * k + a] * Rinv[a * k + b];
  if constexpr (OUT == 0) {
    static_cast<double *>(out)[r * ldo + b] = v;
  } else {
    const bool failed = status[0] != 0 || status[1] != 0;
    if (failed && idx == 0 && err_flag) atomicOr(err_flag, 4);
    if (failed) v = static_cast<double>(U32[r * k + b]);
    if constexpr (OUT == 1)
      static_cast<float *>(out)[r * ldo + b] = static_cast<float>(v);
    else
      static_cast<bf16_t *>(out)[r * ldo + b] = bf16_from_f64(v);
  }
}

template <typename TA, typename TB>
void gram(const TA *A, int64_t lda, const TB *B, int64_t ldb, int64_t d, int64_t k,
          const StepPlan &P, double *partial, double *out, hipStream_t s) {
  gram_partial_kernel<TA, TB><<<dim3(static_cast<unsigned>(P.nch)), 256, 0, s>>>(
      A, lda, B, ldb, d, k, P.rpc, partial);
  gram_reduce_kernel<<<dim3(static_cast<unsigned>(ceil_div(k * k, 256))), 256, 0, s>>>(
      partial, P.nch, k * k, out);
}

}  // namespace

size_t grass_state_bytes(int64_t d, int64_t k) {
  return kGrassStateHead + align256(static_cast<size_t>(d) * k * 8);
}

bool grass_mfma_ok(const PackLayout &L, const void *G, int64_t ldg) {
  return L.mfma && L.d % 64 == 0 && aligned16(G) && ldg % 8 == 0;
}

size_t grass_workspace_bytes(const PackLayout &L, int64_t N) {
  size_t w = acc_plan(L, N, false).total;
  if (L.mfma && L.d % 64 == 0) {
    const size_t m = acc_plan(L, N, true).total;
    w = m > w ? m : w;
  }
  const size_t st = step_plan(L.d, L.k).total;
  return st > w ? st : w;
}

hipError_t launch_grass_reset(void *state, int64_t d, int64_t k, hipStream_t s) {
  const int64_t n = static_cast<int64_t>(grass_state_bytes(d, k) / 8);
  reset_kernel<<<dim3(static_cast<unsigned>(ceil_div(n, 256))), 256, 0, s>>>(
      static_cast<double *>(state), n);
  return hipGetLastError();
}

hipError_t launch_grass_accumulate(const PackLayout &L, const void *packed, const void *G,
                                   int64_t N, int64_t ldg, void *Cwire, int64_t ldc, bool with_su,
                                   void *state, void *ws, hipStream_t s) {
  const char *base = static_cast<const char *>(packed);
  const float *U32 = reinterpret_cast<const float *>(base + L.off_f32);
  char *w = static_cast<char *>(ws);
  double *st = static_cast<double *>(state);
  const bool mfma = grass_mfma_ok(L, G, ldg);
  const AccPlan P = acc_plan(L, N, mfma);
  double *part = reinterpret_cast<double *>(w + P.off_part);
  if (mfma) {
    // the compress writes the loss partials (one per workgroup) and, for Y,
    // the token contraction's operand; the operand's steps past its
    // workgroups (npad > their rows) are zeroed here
    bf16_t *frag = reinterpret_cast<bf16_t *>(w + P.off_frag);
    GrassOut go;
    go.dgram = reinterpret_cast<const double *>(base + L.off_gram);
    go.part = part;
    go.frag = with_su ? frag : nullptr;
    go.nparts = P.nparts;
    go.ktb = P.ktb;
    go.npad = P.npad;
    int64_t steps = 0;
    const int64_t nlblk = grass_compress_groups(L, N, &steps);
    hipError_t e = launch_grass_compress_mfma(L, packed, G, N, ldg, go, Cwire, ldc, s);
    if (e != hipSuccess) return e;
    if (with_su && steps < P.npad / 32) {
      const int64_t per_part = (P.npad / 32) * P.ktb * 512;  // bf16 per operand
      const int64_t tail = (P.npad / 32 - steps) * P.ktb * 512 / 4;  // as doubles
      for (int p = 0; p < P.nparts; ++p) {
        double *t0 = reinterpret_cast<double *>(frag + p * per_part + steps * P.ktb * 512);
        reset_kernel<<<dim3(static_cast<unsigned>(ceil_div(tail, 256))), 256, 0, s>>>(t0, tail);
      }
    }
    float *tp = reinterpret_cast<float *>(w + P.off_tp);
    if (with_su) {
      const int64_t per_part = static_cast<int64_t>(P.npad / 32) * P.ktb * 512;
      for (int p = 0; p < P.nparts; ++p) {
        e = launch_grass_tokens_mfma(frag + p * per_part, P.ktb, P.npad, G, N, ldg, L.d, P.rows,
                                     P.ds, P.m_pad,
                                     tp + static_cast<int64_t>(p) * P.ds * P.m_pad * 16 * P.ktb,
                                     s);
        if (e != hipSuccess) return e;
      }
    }
    const int64_t nfin = with_su ? ceil_div(L.d * L.k, 256) : 1;
    finish_kernel<<<dim3(static_cast<unsigned>(nfin)), 256, 0, s>>>(
        tp, P.ds, P.m_pad, 16 * P.ktb, P.nparts, L.d, L.k, with_su ? 1 : 0, part, nlblk,
        with_su ? 1 : 0, st);
    return hipGetLastError();
  }
  double *C64 = reinterpret_cast<double *>(w + P.off_c);
  const dim3 gc(static_cast<unsigned>(ceil_div(N * L.k, 256)));
  const dim3 gl(static_cast<unsigned>(P.nlblk));
  const dim3 gs(static_cast<unsigned>(ceil_div(L.d * L.k, 256)));
  if (L.dt == 0) {
    const float *g = static_cast<const float *>(G);
    gen_coeff_kernel<float><<<gc, 256, 0, s>>>(g, ldg, U32, N, L.d, L.k, C64);
    gen_loss_kernel<float><<<gl, 256, 0, s>>>(g, ldg, U32, C64, N, L.d, L.k, part);
    if (with_su) gen_su_kernel<float><<<gs, 256, 0, s>>>(g, ldg, C64, N, L.d, L.k, st);
  } else {
    const bf16_t *g = static_cast<const bf16_t *>(G);
    gen_coeff_kernel<bf16_t><<<gc, 256, 0, s>>>(g, ldg, U32, N, L.d, L.k, C64);
    gen_loss_kernel<bf16_t><<<gl, 256, 0, s>>>(g, ldg, U32, C64, N, L.d, L.k, part);
    if (with_su) gen_su_kernel<bf16_t><<<gs, 256, 0, s>>>(g, ldg, C64, N, L.d, L.k, st);
  }
  finish_kernel<<<dim3(1), 256, 0, s>>>(nullptr, 0, 0, 0, 1, L.d, L.k, 0, part, P.nlblk,
                                        with_su ? 1 : 0, st);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  if (Cwire) {
    // the coefficients for the wire, by the kernel the gradient compress uses
    const IdArgs none{};
    if (compress_mfma_ok(L, G, ldg, none))
      return launch_compress_mfma(L, packed, G, N, ldg, none, Cwire, ldc, s);
    return launch_compress_generic(L, packed, G, N, ldg, none, Cwire, ldc, s);
  }
  return hipSuccess;
}

hipError_t launch_grass_step(const PackLayout &L, const void *packed, const void *state,
                             double eta, void *Unew, int64_t ldu, int out_dt, void *ws,
                             int32_t *err_flag, hipStream_t s) {
  const char *base = static_cast<const char *>(packed);
  const float *U32 = reinterpret_cast<const float *>(base + L.off_f32);
  const double *st = static_cast<const double *>(state);
  const double *Y = reinterpret_cast<const double *>(static_cast<const char *>(state) +
                                                     kGrassStateHead);
  const int64_t d = L.d, k = L.k;
  const StepPlan P = step_plan(d, k);
  char *w = static_cast<char *>(ws);
  double *A = reinterpret_cast<double *>(w + P.off_a);
  double *Q = reinterpret_cast<double *>(w + P.off_q);
  double *part = reinterpret_cast<double *>(w + P.off_part);
  double *Z = reinterpret_cast<double *>(w + P.off_z);
  double *Gm = reinterpret_cast<double *>(w + P.off_gram);
  double *R = reinterpret_cast<double *>(w + P.off_r);
  int *status = reinterpret_cast<int *>(w + P.off_status);
  const dim3 gdk(static_cast<unsigned>(ceil_div(d * k, 256)));

  gram<float, double>(U32, k, Y, k, d, k, P, part, Z, s);                 // Z = U^T Y
  update_kernel<<<gdk, 256, 0, s>>>(U32, st, Z, eta, d, k, A, status);    // A = U - eta T
  gram<double, double>(A, k, A, k, d, k, P, part, Gm, s);                 // A^T A
  chol_kernel<<<dim3(1), 256, 0, s>>>(Gm, k, R, status);
  tri_apply_kernel<0><<<gdk, 256, 0, s>>>(A, R, d, k, status, U32, Q, k, nullptr);
  gram<double, double>(Q, k, Q, k, d, k, P, part, Gm, s);                 // Q^T Q
  chol_kernel<<<dim3(1), 256, 0, s>>>(Gm, k, R, status + 1);
  if (out_dt == 0)
    tri_apply_kernel<1><<<gdk, 256, 0, s>>>(Q, R, d, k, status, U32, Unew, ldu, err_flag);
  else
    tri_apply_kernel<2><<<gdk, 256, 0, s>>>(Q, R, d, k, status, U32, Unew, ldu, err_flag);
  return hipGetLastError();
}

}  // namespace sn
