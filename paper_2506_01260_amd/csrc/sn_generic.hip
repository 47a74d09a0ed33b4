// Basis packing and the generic (vector-ALU) codec kernels.
//
// The generic kernels handle every shape, stride and dtype the ABI accepts:
// all float32 work, and bf16 work that does not meet the MFMA kernels'
// alignment / size conditions.  Every sum is a compensated (Dot2) float32
// accumulation, rounded once to the output type, so float32 results stay
// within a few units in the last place even when the sum cancels.
#include "sn_device.h"
#include "sn_internal.h"

namespace sn {

// ---------------------------------------------------------------------------
// Packing
// ---------------------------------------------------------------------------

PackLayout pack_layout(int64_t d, int64_t k, int dt) {
  PackLayout L;
  L.d = d;
  L.k = k;
  L.dt = dt;
  L.kt = static_cast<int>(ceil_div(k, 16));
  L.ks = static_cast<int>(ceil_div(k, 32));
  L.mfma = (dt == 1) && (d % 32 == 0) && (L.kt <= kMfmaMaxKT);
  size_t off = 0;
  L.off_f32 = off;
  off = align256(off + static_cast<size_t>(d) * k * 4);
  if (L.mfma) {
    L.off_kfrag = off;
    off = align256(off + static_cast<size_t>(d / 32) * L.kt * 1024);
    L.off_rfrag = off;
    off = align256(off + static_cast<size_t>(d / 32) * 2 * L.ks * 1024);
    if (k <= 64) {
      L.ks2 = static_cast<int>(ceil_div(2 * k, 32));
      L.off_uu = off;
      off = align256(off + static_cast<size_t>(d) * 32 * L.ks2 * 2);
    }
  }
  L.off_gram = off;
  off = align256(off + static_cast<size_t>(16 * L.kt) * (16 * L.kt) * 8);
  L.total = off;
  return L;
}

template <typename T>
__global__ __launch_bounds__(256) void pack_f32_kernel(const T *__restrict__ U, int64_t d,
                                                       int64_t k, int64_t ldu,
                                                       float *__restrict__ out) {
  int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= d * k) return;
  int64_t r = idx / k, j = idx - r * k;
  out[idx] = to_f32(U[r * ldu + j]);
}

// One thread per 8-element lane slot of a 1 KiB fragment block.
__global__ __launch_bounds__(256) void pack_kfrag_kernel(const bf16_t *__restrict__ U, int64_t d,
                                                         int64_t k, int64_t ldu, int kt,
                                                         bf16_t *__restrict__ out) {
  int64_t slot = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;  // (block, lane)
  int64_t nblk = (d / 32) * kt;
  if (slot >= nblk * 64) return;
  int64_t blk = slot >> 6;
  int lane = static_cast<int>(slot & 63);
  int64_t s = blk / kt;
  int t = static_cast<int>(blk - s * kt);
  int g = lane >> 4, n = lane & 15;
  int64_t col = 16 * t + n;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    int64_t row = 32 * s + 8 * g + e;
    out[slot * 8 + e] = col < k ? U[row * ldu + col] : bf16_t(0);
  }
}

__global__ __launch_bounds__(256) void pack_rfrag_kernel(const bf16_t *__restrict__ U, int64_t d,
                                                         int64_t k, int64_t ldu, int ks,
                                                         bf16_t *__restrict__ out) {
  int64_t slot = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  int64_t nblk = (d / 32) * 2 * ks;
  if (slot >= nblk * 64) return;
  int64_t blk = slot >> 6;
  int lane = static_cast<int>(slot & 63);
  int q = static_cast<int>(blk % ks);
  int h = static_cast<int>((blk / ks) & 1);
  int64_t p = blk / (2 * ks);
  int g = lane >> 4, m = lane & 15;
  int64_t row = 32 * p + 8 * (m >> 2) + 4 * h + (m & 3);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    int64_t col = 32 * q + 8 * g + e;
    out[slot * 8 + e] = col < k ? U[row * ldu + col] : bf16_t(0);
  }
}

// [U | U] with zero columns up to 32 ks2, one thread per element.
__global__ __launch_bounds__(256) void pack_uu_kernel(const bf16_t *__restrict__ U, int64_t d,
                                                      int64_t k, int64_t ldu, int ks2,
                                                      bf16_t *__restrict__ out) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int w = 32 * ks2;
  if (idx >= d * w) return;
  const int64_t r = idx / w;
  const int64_t j = idx - r * w;
  out[idx] = j < 2 * k ? U[r * ldu + (j < k ? j : j - k)] : bf16_t(0);
}

// U^T U - I from the float32 section (exact copies of the stored U), as a
// kp x kp matrix (kp = 16 ceil(k/16) <= 256, zero outside k x k).  One
// workgroup per row a; thread (h, b) sums U[r, a] U[r, b] in float64 over the
// rows r = h mod H (H = 1024 / kp row phases, reads coalesced along b), and
// the H partial sums are added in a fixed order.
constexpr int kGramThreads = 1024;
__global__ __launch_bounds__(kGramThreads) void pack_gram_kernel(const float *__restrict__ U32,
                                                                 int64_t d, int64_t k, int64_t kp,
                                                                 double *__restrict__ out) {
  __shared__ double red[kGramThreads];
  const int64_t a = blockIdx.x;
  const int H = static_cast<int>(kGramThreads / kp);
  const int h = static_cast<int>(threadIdx.x / kp), b = static_cast<int>(threadIdx.x % kp);
  double acc = 0.0;
  if (a < k && h < H && b < k) {
#pragma unroll 4
    for (int64_t r = h; r < d; r += H)
      acc += static_cast<double>(U32[r * k + a]) * static_cast<double>(U32[r * k + b]);
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x < kp) {
    double v = 0.0;
    for (int hh = 0; hh < H; ++hh) v += red[hh * kp + threadIdx.x];
    const bool in = a < k && static_cast<int64_t>(threadIdx.x) < k;
    out[a * kp + threadIdx.x] = in ? v - (a == static_cast<int64_t>(threadIdx.x) ? 1.0 : 0.0)
                                   : 0.0;
  }
}

hipError_t launch_pack(const PackLayout &L, const void *U, int64_t ldu, void *packed,
                       hipStream_t s) {
  char *base = static_cast<char *>(packed);
  int64_t n = L.d * L.k;
  dim3 grid(static_cast<unsigned>(ceil_div(n, 256)));
  if (L.dt == 0)
    pack_f32_kernel<float><<<grid, 256, 0, s>>>(static_cast<const float *>(U), L.d, L.k, ldu,
                                                reinterpret_cast<float *>(base + L.off_f32));
  else
    pack_f32_kernel<bf16_t><<<grid, 256, 0, s>>>(static_cast<const bf16_t *>(U), L.d, L.k, ldu,
                                                 reinterpret_cast<float *>(base + L.off_f32));
  if (L.mfma) {
    const bf16_t *Ub = static_cast<const bf16_t *>(U);
    int64_t slots = (L.d / 32) * L.kt * 64;
    pack_kfrag_kernel<<<dim3(static_cast<unsigned>(ceil_div(slots, 256))), 256, 0, s>>>(
        Ub, L.d, L.k, ldu, L.kt, reinterpret_cast<bf16_t *>(base + L.off_kfrag));
    slots = (L.d / 32) * 2 * L.ks * 64;
    pack_rfrag_kernel<<<dim3(static_cast<unsigned>(ceil_div(slots, 256))), 256, 0, s>>>(
        Ub, L.d, L.k, ldu, L.ks, reinterpret_cast<bf16_t *>(base + L.off_rfrag));
    if (L.ks2 > 0) {
      const int64_t nu = L.d * 32 * L.ks2;
      pack_uu_kernel<<<dim3(static_cast<unsigned>(ceil_div(nu, 256))), 256, 0, s>>>(
          Ub, L.d, L.k, ldu, L.ks2, reinterpret_cast<bf16_t *>(base + L.off_uu));
    }
  }
  const int64_t kp = 16 * L.kt;
  pack_gram_kernel<<<dim3(static_cast<unsigned>(kp)), kGramThreads, 0, s>>>(
      reinterpret_cast<const float *>(base + L.off_f32), L.d, L.k, kp,
      reinterpret_cast<double *>(base + L.off_gram));
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Token / position row resolution shared by the generic kernels
// ---------------------------------------------------------------------------

template <typename T>
struct Rows {
  const T *e;  // T_fixed row of the token, or nullptr
  const T *p;  // positional row, or nullptr
};

template <typename T>
__device__ __forceinline__ Rows<T> resolve_rows(int64_t i, const IdArgs &a) {
  Rows<T> r{nullptr, nullptr};
  if (a.E) {
    int64_t t = clamp_id(a.tok[i], a.vocab, a.err_flag, 1);
    r.e = static_cast<const T *>(a.E) + t * a.lde;
  }
  if (a.P) {
    int64_t p = a.pos ? static_cast<int64_t>(a.pos[i]) : i % a.seq_len;
    p = clamp_id(p, a.n_pos, a.err_flag, 2);
    r.p = static_cast<const T *>(a.P) + p * a.ldp;
  }
  return r;
}

// ---------------------------------------------------------------------------
// Compress: one wave per token.  Each lane strides over d, accumulates up to
// 8 columns of C at a time, and the wave reduces with cross-lane shuffles.
// ---------------------------------------------------------------------------

template <typename T>
__global__ __launch_bounds__(256) void compress_generic_kernel(const float *__restrict__ Uf,
                                                               int64_t d, int64_t k,
                                                               const T *__restrict__ X,
                                                               int64_t N, int64_t ldx, IdArgs ids,
                                                               T *__restrict__ C, int64_t ldc) {
  const int lane = threadIdx.x & 63;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (i >= N) return;
  const Rows<T> rw = resolve_rows<T>(i, ids);
  const T *xr = X + i * ldx;
  // (X - P - E) U is summed as X U - P U - E U: no rounding of X - P - E.
  for (int64_t j0 = 0; j0 < k; j0 += 8) {
    Dot2 acc[8];
    const int jn = static_cast<int>(k - j0 < 8 ? k - j0 : 8);
    for (int64_t r = lane; r < d; r += 64) {
      const float x = to_f32(xr[r]);
      const float p = rw.p ? -to_f32(rw.p[r]) : 0.0f;
      const float e = rw.e ? -to_f32(rw.e[r]) : 0.0f;
      const float *ur = Uf + r * k + j0;
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        if (jj < jn) {
          acc[jj].add_prod(x, ur[jj]);
          if (rw.p) acc[jj].add_prod(p, ur[jj]);
          if (rw.e) acc[jj].add_prod(e, ur[jj]);
        }
      }
    }
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      const float v = wave_sum_dot2(acc[jj]);
      if (lane == 0 && jj < jn) C[i * ldc + j0 + jj] = from_f32<T>(v);
    }
  }
}

hipError_t launch_compress_generic(const PackLayout &L, const void *packed, const void *X,
                                   int64_t N, int64_t ldx, const IdArgs &ids, void *C,
                                   int64_t ldc, hipStream_t s) {
  const float *Uf = reinterpret_cast<const float *>(static_cast<const char *>(packed) + L.off_f32);
  dim3 grid(static_cast<unsigned>(ceil_div(N, 4)));
  if (L.dt == 0)
    compress_generic_kernel<float><<<grid, 256, 0, s>>>(
        Uf, L.d, L.k, static_cast<const float *>(X), N, ldx, ids, static_cast<float *>(C), ldc);
  else
    compress_generic_kernel<bf16_t><<<grid, 256, 0, s>>>(
        Uf, L.d, L.k, static_cast<const bf16_t *>(X), N, ldx, ids, static_cast<bf16_t *>(C), ldc);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Projected tables and compress against them (one wave per row, as above).
// TABLE: out[r, j] = (T U)[r, j] as fp32 for j < k, 0 for k <= j < kp.
// Otherwise: C[i, j] = (X U)[i, j] - (P U)[pos_i, j] - (T_fixed U)[tok_i, j],
// each subtraction rounded to fp32, then one rounding to the output type.
// ---------------------------------------------------------------------------

ProjLayout proj_layout(int64_t k, int64_t vocab, int64_t n_pos) {
  ProjLayout P;
  P.kp = 16 * ceil_div(k, 16);
  P.off_eu = 0;
  P.off_pu = align256(static_cast<size_t>(vocab) * P.kp * sizeof(float));
  P.total = P.off_pu + align256(static_cast<size_t>(n_pos) * P.kp * sizeof(float));
  return P;
}

template <typename T, bool TABLE>
__global__ __launch_bounds__(256) void project_rows_generic_kernel(
    const float *__restrict__ Uf, int64_t d, int64_t k, const T *__restrict__ X, int64_t N,
    int64_t ldx, ProjArgs pa, void *__restrict__ out, int64_t ldo) {
  const int lane = threadIdx.x & 63;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (i >= N) return;
  const T *xr = X + i * ldx;
  const float *pr = nullptr, *er = nullptr;
  if (!TABLE) {
    if (pa.pu) {
      int64_t p = pa.pos ? static_cast<int64_t>(pa.pos[i]) : i % pa.seq_len;
      pr = pa.pu + clamp_id(p, pa.n_pos, pa.err_flag, 2) * pa.kp;
    }
    if (pa.eu) er = pa.eu + clamp_id(pa.tok[i], pa.vocab, pa.err_flag, 1) * pa.kp;
  }
  const int64_t ncols = TABLE ? ldo : k;  // a table row is written out to its padded width
  for (int64_t j0 = 0; j0 < ncols; j0 += 8) {
    Dot2 acc[8];
    const int jn = static_cast<int>(k - j0 < 8 ? (k - j0 > 0 ? k - j0 : 0) : 8);
    for (int64_t r = lane; r < d && jn > 0; r += 64) {
      const float x = to_f32(xr[r]);
      const float *ur = Uf + r * k + j0;
#pragma unroll
      for (int jj = 0; jj < 8; ++jj)
        if (jj < jn) acc[jj].add_prod(x, ur[jj]);
    }
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      float v = wave_sum_dot2(acc[jj]);
      const int64_t j = j0 + jj;
      if (lane != 0) continue;
      if (TABLE) {
        if (j < ncols) static_cast<float *>(out)[i * ldo + j] = jj < jn ? v : 0.0f;
      } else if (jj < jn) {
        if (pr) v = __fsub_rn(v, pr[j]);
        if (er) v = __fsub_rn(v, er[j]);
        static_cast<T *>(out)[i * ldo + j] = from_f32<T>(v);
      }
    }
  }
}

hipError_t launch_table_project_generic(const PackLayout &L, const void *packed, const void *T,
                                        int64_t rows, int64_t ldt, float *out, int64_t kp,
                                        hipStream_t s) {
  const float *Uf = reinterpret_cast<const float *>(static_cast<const char *>(packed) + L.off_f32);
  dim3 grid(static_cast<unsigned>(ceil_div(rows, 4)));
  ProjArgs none{};
  if (L.dt == 0)
    project_rows_generic_kernel<float, true><<<grid, 256, 0, s>>>(
        Uf, L.d, L.k, static_cast<const float *>(T), rows, ldt, none, out, kp);
  else
    project_rows_generic_kernel<bf16_t, true><<<grid, 256, 0, s>>>(
        Uf, L.d, L.k, static_cast<const bf16_t *>(T), rows, ldt, none, out, kp);
  return hipGetLastError();
}

hipError_t launch_compress_projected_generic(const PackLayout &L, const void *packed,
                                             const void *X, int64_t N, int64_t ldx,
                                             const ProjArgs &pa, void *C, int64_t ldc,
                                             hipStream_t s) {
  const float *Uf = reinterpret_cast<const float *>(static_cast<const char *>(packed) + L.off_f32);
  dim3 grid(static_cast<unsigned>(ceil_div(N, 4)));
  if (L.dt == 0)
    project_rows_generic_kernel<float, false><<<grid, 256, 0, s>>>(
        Uf, L.d, L.k, static_cast<const float *>(X), N, ldx, pa, C, ldc);
  else
    project_rows_generic_kernel<bf16_t, false><<<grid, 256, 0, s>>>(
        Uf, L.d, L.k, static_cast<const bf16_t *>(X), N, ldx, pa, C, ldc);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Decompress: one thread per output element; blockIdx.x = token,
// blockIdx.y = 256-wide slice of d.
// ---------------------------------------------------------------------------

template <typename T>
__global__ __launch_bounds__(256) void decompress_generic_kernel(const float *__restrict__ Uf,
                                                                 int64_t d, int64_t k,
                                                                 const T *__restrict__ C,
                                                                 int64_t ldc, IdArgs ids,
                                                                 T *__restrict__ X, int64_t ldx) {
  const int64_t i = blockIdx.x;
  const int64_t r = static_cast<int64_t>(blockIdx.y) * 256 + threadIdx.x;
  if (r >= d) return;
  const Rows<T> rw = resolve_rows<T>(i, ids);
  const T *cr = C + i * ldc;
  const float *ur = Uf + r * k;
  Dot2 acc;
  for (int64_t j = 0; j < k; ++j) acc.add_prod(to_f32(cr[j]), ur[j]);
  if (rw.p) acc.add(to_f32(rw.p[r]));
  if (rw.e) acc.add(to_f32(rw.e[r]));
  X[i * ldx + r] = from_f32<T>(acc.value());
}

hipError_t launch_decompress_generic(const PackLayout &L, const void *packed, const void *C,
                                     int64_t N, int64_t ldc, const IdArgs &ids, void *X,
                                     int64_t ldx, hipStream_t s) {
  const float *Uf = reinterpret_cast<const float *>(static_cast<const char *>(packed) + L.off_f32);
  const int64_t ychunks = ceil_div(L.d, 256);
  // gridDim.x holds the tokens (up to 2^31-1), gridDim.y the d slices.
  dim3 grid(static_cast<unsigned>(N), static_cast<unsigned>(ychunks));
  if (L.dt == 0)
    decompress_generic_kernel<float><<<grid, 256, 0, s>>>(
        Uf, L.d, L.k, static_cast<const float *>(C), ldc, ids, static_cast<float *>(X), ldx);
  else
    decompress_generic_kernel<bf16_t><<<grid, 256, 0, s>>>(
        Uf, L.d, L.k, static_cast<const bf16_t *>(C), ldc, ids, static_cast<bf16_t *>(X), ldx);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight projection W <- U (U^T W), generic path, three passes:
//   1. partial T_s = U[rows of split s]^T W[rows of split s]   (fp32, per split)
//   2. T = sum_s T_s in fixed split order
//   3. W[r, c] = sum_j U[r, j] T[j, c]
// Workspace: S * k * m floats of partials followed by k * m floats of T.
// ---------------------------------------------------------------------------

constexpr int kGenericRowsPerSplit = 256;

inline int64_t generic_splits(int64_t d) {
  int64_t s = ceil_div(d, kGenericRowsPerSplit);
  return s > 64 ? 64 : s;
}

size_t project_workspace_generic(int64_t d, int64_t k, int64_t m) {
  return static_cast<size_t>(generic_splits(d) + 1) * k * m * sizeof(float);
}

template <typename T>
__global__ __launch_bounds__(256) void project_partial_kernel(const float *__restrict__ Uf,
                                                              int64_t d, int64_t k,
                                                              const T *__restrict__ W, int64_t m,
                                                              int64_t ldw, int64_t rows_per_split,
                                                              float *__restrict__ Tp) {
  const int64_t c = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (c >= m) return;
  const int64_t s = blockIdx.y;
  const int64_t r0 = s * rows_per_split;
  const int64_t r1 = r0 + rows_per_split < d ? r0 + rows_per_split : d;
  for (int64_t j0 = 0; j0 < k; j0 += 8) {
    Dot2 acc[8];
    const int jn = static_cast<int>(k - j0 < 8 ? k - j0 : 8);
    for (int64_t r = r0; r < r1; ++r) {
      const float w = to_f32(W[r * ldw + c]);
      const float *ur = Uf + r * k + j0;
#pragma unroll
      for (int jj = 0; jj < 8; ++jj)
        if (jj < jn) acc[jj].add_prod(ur[jj], w);
    }
#pragma unroll
    for (int jj = 0; jj < 8; ++jj)
      if (jj < jn) Tp[(s * k + j0 + jj) * m + c] = acc[jj].value();
  }
}

__global__ __launch_bounds__(256) void project_reduce_kernel(const float *__restrict__ Tp,
                                                             int64_t splits, int64_t km,
                                                             float *__restrict__ T) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= km) return;
  Dot2 acc;
  for (int64_t s = 0; s < splits; ++s) acc.add(Tp[s * km + idx]);
  T[idx] = acc.value();
}

template <typename T>
__global__ __launch_bounds__(256) void project_expand_kernel(const float *__restrict__ Uf,
                                                             int64_t k, const float *__restrict__ Tm,
                                                             T *__restrict__ W, int64_t m,
                                                             int64_t ldw, int64_t cblocks) {
  // blockIdx.x = r * cblocks + (256-column block)
  const int64_t r = blockIdx.x / cblocks;
  const int64_t c = (blockIdx.x - r * cblocks) * 256 + threadIdx.x;
  if (c >= m) return;
  const float *ur = Uf + r * k;
  Dot2 acc;
  for (int64_t j = 0; j < k; ++j) acc.add_prod(ur[j], Tm[j * m + c]);
  W[r * ldw + c] = from_f32<T>(acc.value());
}

hipError_t launch_project_generic(const PackLayout &L, const void *packed, void *W, int64_t m,
                                  int64_t ldw, void *ws, hipStream_t s) {
  const float *Uf = reinterpret_cast<const float *>(static_cast<const char *>(packed) + L.off_f32);
  const int64_t S = generic_splits(L.d);
  const int64_t rps = ceil_div(L.d, S);
  float *Tp = static_cast<float *>(ws);
  float *Tm = Tp + S * L.k * m;
  dim3 g1(static_cast<unsigned>(ceil_div(m, 256)), static_cast<unsigned>(S));
  const int64_t km = L.k * m;
  dim3 g2(static_cast<unsigned>(ceil_div(km, 256)));
  const int64_t cblocks = ceil_div(m, 256);
  dim3 g3(static_cast<unsigned>(cblocks * L.d));
  if (L.dt == 0) {
    project_partial_kernel<float><<<g1, 256, 0, s>>>(Uf, L.d, L.k, static_cast<const float *>(W),
                                                     m, ldw, rps, Tp);
    project_reduce_kernel<<<g2, 256, 0, s>>>(Tp, S, km, Tm);
    project_expand_kernel<float><<<g3, 256, 0, s>>>(Uf, L.k, Tm, static_cast<float *>(W), m, ldw,
                                                    cblocks);
  } else {
    project_partial_kernel<bf16_t><<<g1, 256, 0, s>>>(Uf, L.d, L.k,
                                                      static_cast<const bf16_t *>(W), m, ldw,
                                                      rps, Tp);
    project_reduce_kernel<<<g2, 256, 0, s>>>(Tp, S, km, Tm);
    project_expand_kernel<bf16_t><<<g3, 256, 0, s>>>(Uf, L.k, Tm, static_cast<bf16_t *>(W), m,
                                                     ldw, cblocks);
  }
  return hipGetLastError();
}

}  // namespace sn
