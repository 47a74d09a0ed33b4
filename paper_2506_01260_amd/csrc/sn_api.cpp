// The C ABI: host-side argument validation and dispatch to the kernels.
// Every check runs before anything is launched; see include/sn.h for the
// contract of each entry point.
#include "sn.h"

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "sn_internal.h"

namespace {

thread_local char g_err[512] = "";

int32_t fail(int32_t st, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

int32_t ok() {
  g_err[0] = '\0';
  return SN_OK;
}

}  // namespace


namespace sn {

int32_t set_error(int32_t st, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

}  // namespace sn

namespace {

int32_t hip_status(hipError_t e, const char *what) {
  if (e == hipSuccess) return ok();
  return fail(SN_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

size_t elem_size(int32_t dt) { return dt == SN_F32 ? 4 : 2; }

bool dtype_ok(int32_t dt) { return dt == SN_F32 || dt == SN_BF16; }

bool elem_aligned(const void *p, int32_t dt) {
  return (reinterpret_cast<uintptr_t>(p) & (elem_size(dt) - 1)) == 0;
}

// Byte range [lo, hi) covered by a rows x cols matrix with row stride ld.
struct Span {
  uintptr_t lo = 0, hi = 0;
};

Span span(const void *p, int64_t rows, int64_t cols, int64_t ld, size_t es) {
  Span s;
  if (!p || rows <= 0 || cols <= 0) return s;
  s.lo = reinterpret_cast<uintptr_t>(p);
  s.hi = s.lo + (static_cast<uintptr_t>(rows - 1) * ld + cols) * es;
  return s;
}

bool overlap(Span a, Span b) { return a.lo < a.hi && b.lo < b.hi && a.lo < b.hi && b.lo < a.hi; }

constexpr int64_t kMaxDim = int64_t(1) << 31;  // rows, columns and strides stay below 2^31

int32_t check_basis(const void *basis, int64_t d, int64_t k, int32_t dt) {
  if (!dtype_ok(dt)) return fail(SN_ERR_DTYPE, "unknown dtype %d", dt);
  if (!basis) return fail(SN_ERR_NULL, "basis is NULL");
  if (reinterpret_cast<uintptr_t>(basis) & 255)
    return fail(SN_ERR_ALIGN, "packed basis must be 256-byte aligned");
  if (d < 1 || d >= kMaxDim) return fail(SN_ERR_SHAPE, "d = %lld out of range", (long long)d);
  if (k < 1 || k > d) return fail(SN_ERR_SHAPE, "k = %lld must satisfy 1 <= k <= d", (long long)k);
  if (k > SN_MAX_K) return fail(SN_ERR_UNSUPPORTED, "k = %lld > SN_MAX_K", (long long)k);
  return SN_OK;
}

// Validates the id / table arguments shared by compress and decompress.
int32_t check_ids(int64_t N, int64_t d, int32_t dt, const int32_t *tok, const void *E,
                  int64_t vocab, int64_t lde, const int32_t *pos, const void *P, int64_t n_pos,
                  int64_t ldp, int64_t seq_len) {
  if (E) {
    if (vocab < 1 || vocab >= kMaxDim)
      return fail(SN_ERR_SHAPE, "vocab = %lld out of range", (long long)vocab);
    if (lde < d || lde >= kMaxDim) return fail(SN_ERR_SHAPE, "lde must be >= d");
    if (N > 0 && !tok) return fail(SN_ERR_NULL, "tok is NULL but E is given");
    if (!elem_aligned(E, dt)) return fail(SN_ERR_ALIGN, "E not aligned to its element size");
    if (tok && (reinterpret_cast<uintptr_t>(tok) & 3))
      return fail(SN_ERR_ALIGN, "tok not 4-byte aligned");
  }
  if (P) {
    if (n_pos < 1 || n_pos >= kMaxDim)
      return fail(SN_ERR_SHAPE, "n_pos = %lld out of range", (long long)n_pos);
    if (ldp < d || ldp >= kMaxDim) return fail(SN_ERR_SHAPE, "ldp must be >= d");
    if (!pos && (seq_len < 1 || seq_len > n_pos))
      return fail(SN_ERR_SHAPE, "pos is NULL: need 1 <= seq_len <= n_pos (seq_len = %lld)",
                  (long long)seq_len);
    if (!elem_aligned(P, dt)) return fail(SN_ERR_ALIGN, "P not aligned to its element size");
    if (pos && (reinterpret_cast<uintptr_t>(pos) & 3))
      return fail(SN_ERR_ALIGN, "pos not 4-byte aligned");
  }
  return SN_OK;
}

// The output span must not overlap any input span.
int32_t check_out_alias(Span out, const void *basis, size_t basis_bytes, Span in, int64_t N,
                        const int32_t *tok, const void *E, int64_t vocab, int64_t lde,
                        const int32_t *pos, const void *P, int64_t n_pos, int64_t ldp,
                        int64_t d, size_t es) {
  Span b;
  b.lo = reinterpret_cast<uintptr_t>(basis);
  b.hi = b.lo + basis_bytes;
  if (overlap(out, b)) return fail(SN_ERR_ALIAS, "output overlaps the packed basis");
  if (overlap(out, in)) return fail(SN_ERR_ALIAS, "output overlaps the input matrix");
  if (E && overlap(out, span(E, vocab, d, lde, es)))
    return fail(SN_ERR_ALIAS, "output overlaps E");
  if (P && overlap(out, span(P, n_pos, d, ldp, es)))
    return fail(SN_ERR_ALIAS, "output overlaps P");
  if (E && tok && overlap(out, span(tok, 1, N, N, 4)))
    return fail(SN_ERR_ALIAS, "output overlaps tok");
  if (P && pos && overlap(out, span(pos, 1, N, N, 4)))
    return fail(SN_ERR_ALIAS, "output overlaps pos");
  return SN_OK;
}

Span bytes_span(const void *p, size_t n) {
  Span s;
  if (!p || n == 0) return s;
  s.lo = reinterpret_cast<uintptr_t>(p);
  s.hi = s.lo + n;
  return s;
}

int32_t check_state(const void *state, int64_t d, int64_t k) {
  if (!state) return fail(SN_ERR_NULL, "state is NULL");
  if (reinterpret_cast<uintptr_t>(state) & 255)
    return fail(SN_ERR_ALIGN, "state must be 256-byte aligned");
  if (k > sn::kGrassMaxK)
    return fail(SN_ERR_UNSUPPORTED, "subspace update needs k <= %d", sn::kGrassMaxK);
  (void)d;
  return SN_OK;
}

int32_t check_workspace(const void *ws, size_t have, size_t need) {
  if (!ws) return fail(SN_ERR_NULL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) & 255)
    return fail(SN_ERR_ALIGN, "workspace must be 256-byte aligned");
  if (have < need) return fail(SN_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", have, need);
  return SN_OK;
}

sn::IdArgs make_ids(const int32_t *tok, const void *E, int64_t vocab, int64_t lde,
                    const int32_t *pos, const void *P, int64_t n_pos, int64_t ldp,
                    int64_t seq_len, int32_t *err_flag) {
  sn::IdArgs a;
  a.E = E;
  a.tok = E ? tok : nullptr;
  a.vocab = vocab;
  a.lde = lde;
  a.P = P;
  a.pos = P ? pos : nullptr;
  a.n_pos = n_pos;
  a.ldp = ldp;
  a.seq_len = (P && !pos) ? seq_len : 1;
  a.err_flag = err_flag;
  return a;
}

}  // namespace

namespace sn {

int32_t project_args_check(const void *basis, int64_t d, int64_t k, int32_t dt, const void *W,
                           int64_t m, int64_t ldw) {
  int32_t st = check_basis(basis, d, k, dt);
  if (st) return st;
  if (m < 0 || m >= kMaxDim) return fail(SN_ERR_SHAPE, "m out of range");
  if (ldw < m || ldw >= kMaxDim) return fail(SN_ERR_SHAPE, "ldw must be >= m");
  if (m == 0) return ok();
  if (!W) return fail(SN_ERR_NULL, "W is NULL");
  if (!elem_aligned(W, dt)) return fail(SN_ERR_ALIGN, "W not aligned to its element size");
  return ok();
}

}  // namespace sn

extern "C" {

size_t sn_basis_packed_bytes(int64_t d, int64_t k, int32_t dt) {
  if (!dtype_ok(dt) || d < 1 || d >= kMaxDim || k < 1 || k > d || k > SN_MAX_K) return 0;
  return sn::pack_layout(d, k, dt).total;
}

int32_t sn_basis_pack(const void *U, int64_t d, int64_t k, int64_t ldu, int32_t dt, void *packed,
                      size_t packed_bytes, sn_stream stream) {
  if (!dtype_ok(dt)) return fail(SN_ERR_DTYPE, "unknown dtype %d", dt);
  if (!U || !packed) return fail(SN_ERR_NULL, "U or packed is NULL");
  if (d < 1 || d >= kMaxDim) return fail(SN_ERR_SHAPE, "d out of range");
  if (k < 1 || k > d) return fail(SN_ERR_SHAPE, "need 1 <= k <= d");
  if (k > SN_MAX_K) return fail(SN_ERR_UNSUPPORTED, "k > SN_MAX_K");
  if (ldu < k || ldu >= kMaxDim) return fail(SN_ERR_SHAPE, "ldu must be >= k");
  if (!elem_aligned(U, dt)) return fail(SN_ERR_ALIGN, "U not aligned to its element size");
  if (reinterpret_cast<uintptr_t>(packed) & 255)
    return fail(SN_ERR_ALIGN, "packed must be 256-byte aligned");
  const sn::PackLayout L = sn::pack_layout(d, k, dt);
  if (packed_bytes < L.total)
    return fail(SN_ERR_WORKSPACE, "packed buffer has %zu bytes, needs %zu", packed_bytes, L.total);
  Span pu;
  pu.lo = reinterpret_cast<uintptr_t>(packed);
  pu.hi = pu.lo + L.total;
  if (overlap(pu, span(U, d, k, ldu, elem_size(dt))))
    return fail(SN_ERR_ALIAS, "packed overlaps U");
  return hip_status(sn::launch_pack(L, U, ldu, packed, static_cast<hipStream_t>(stream)),
                    "sn_basis_pack launch");
}

int32_t sn_compress(const void *basis, int64_t d, int64_t k, int32_t dt, const void *X, int64_t N,
                    int64_t ldx, const int32_t *tok, const void *E, int64_t vocab, int64_t lde,
                    const int32_t *pos, const void *P, int64_t n_pos, int64_t ldp,
                    int64_t seq_len, void *C, int64_t ldc, int32_t *err_flag, sn_stream stream) {
  int32_t st = check_basis(basis, d, k, dt);
  if (st) return st;
  if (N < 0 || N >= kMaxDim) return fail(SN_ERR_SHAPE, "N = %lld out of range", (long long)N);
  if (ldx < d || ldx >= kMaxDim) return fail(SN_ERR_SHAPE, "ldx must be >= d");
  if (ldc < k || ldc >= kMaxDim) return fail(SN_ERR_SHAPE, "ldc must be >= k");
  if ((st = check_ids(N, d, dt, tok, E, vocab, lde, pos, P, n_pos, ldp, seq_len))) return st;
  if (N == 0) return ok();
  if (!X || !C) return fail(SN_ERR_NULL, "X or C is NULL");
  if (!elem_aligned(X, dt) || !elem_aligned(C, dt))
    return fail(SN_ERR_ALIGN, "X or C not aligned to its element size");
  const size_t es = elem_size(dt);
  const sn::PackLayout L = sn::pack_layout(d, k, dt);
  if ((st = check_out_alias(span(C, N, k, ldc, es), basis, L.total, span(X, N, d, ldx, es), N,
                            tok, E, vocab, lde, pos, P, n_pos, ldp, d, es)))
    return st;
  const sn::IdArgs ids = make_ids(tok, E, vocab, lde, pos, P, n_pos, ldp, seq_len, err_flag);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (sn::compress_mfma_ok(L, X, ldx, ids))
    return hip_status(sn::launch_compress_mfma(L, basis, X, N, ldx, ids, C, ldc, s),
                      "sn_compress launch");
  return hip_status(sn::launch_compress_generic(L, basis, X, N, ldx, ids, C, ldc, s),
                    "sn_compress launch");
}

int32_t sn_decompress(const void *basis, int64_t d, int64_t k, int32_t dt, const void *C,
                      int64_t N, int64_t ldc, const int32_t *tok, const void *E, int64_t vocab,
                      int64_t lde, const int32_t *pos, const void *P, int64_t n_pos, int64_t ldp,
                      int64_t seq_len, void *X, int64_t ldx, int32_t *err_flag,
                      sn_stream stream) {
  int32_t st = check_basis(basis, d, k, dt);
  if (st) return st;
  if (N < 0 || N >= kMaxDim) return fail(SN_ERR_SHAPE, "N = %lld out of range", (long long)N);
  if (ldx < d || ldx >= kMaxDim) return fail(SN_ERR_SHAPE, "ldx must be >= d");
  if (ldc < k || ldc >= kMaxDim) return fail(SN_ERR_SHAPE, "ldc must be >= k");
  if ((st = check_ids(N, d, dt, tok, E, vocab, lde, pos, P, n_pos, ldp, seq_len))) return st;
  if (N == 0) return ok();
  if (!X || !C) return fail(SN_ERR_NULL, "X or C is NULL");
  if (!elem_aligned(X, dt) || !elem_aligned(C, dt))
    return fail(SN_ERR_ALIGN, "X or C not aligned to its element size");
  const size_t es = elem_size(dt);
  const sn::PackLayout L = sn::pack_layout(d, k, dt);
  if ((st = check_out_alias(span(X, N, d, ldx, es), basis, L.total, span(C, N, k, ldc, es), N,
                            tok, E, vocab, lde, pos, P, n_pos, ldp, d, es)))
    return st;
  const sn::IdArgs ids = make_ids(tok, E, vocab, lde, pos, P, n_pos, ldp, seq_len, err_flag);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (sn::decompress_mfma_ok(L, X, ldx, ids))
    return hip_status(sn::launch_decompress_mfma(L, basis, C, N, ldc, ids, X, ldx, s),
                      "sn_decompress launch");
  return hip_status(sn::launch_decompress_generic(L, basis, C, N, ldc, ids, X, ldx, s),
                    "sn_decompress launch");
}

int32_t sn_grad_compress(const void *basis, int64_t d, int64_t k, int32_t dt, const void *G,
                         int64_t N, int64_t ldg, void *Cg, int64_t ldc, sn_stream stream) {
  return sn_compress(basis, d, k, dt, G, N, ldg, nullptr, nullptr, 0, 0, nullptr, nullptr, 0, 0,
                     0, Cg, ldc, nullptr, stream);
}

size_t sn_embed_projected_bytes(int64_t k, int64_t vocab, int64_t n_pos) {
  if (k < 1 || k > SN_MAX_K || vocab < 0 || vocab >= kMaxDim || n_pos < 0 || n_pos >= kMaxDim)
    return 0;
  return sn::proj_layout(k, vocab, n_pos).total;
}

int32_t sn_embed_project(const void *basis, int64_t d, int64_t k, int32_t dt, const void *E,
                         int64_t vocab, int64_t lde, const void *P, int64_t n_pos, int64_t ldp,
                         void *proj, size_t proj_bytes, sn_stream stream) {
  int32_t st = check_basis(basis, d, k, dt);
  if (st) return st;
  if (vocab < 0 || vocab >= kMaxDim) return fail(SN_ERR_SHAPE, "vocab out of range");
  if (n_pos < 0 || n_pos >= kMaxDim) return fail(SN_ERR_SHAPE, "n_pos out of range");
  if ((vocab > 0) != (E != nullptr)) return fail(SN_ERR_NULL, "E must be given iff vocab > 0");
  if ((n_pos > 0) != (P != nullptr)) return fail(SN_ERR_NULL, "P must be given iff n_pos > 0");
  if (E && (lde < d || lde >= kMaxDim)) return fail(SN_ERR_SHAPE, "lde must be >= d");
  if (P && (ldp < d || ldp >= kMaxDim)) return fail(SN_ERR_SHAPE, "ldp must be >= d");
  if ((E && !elem_aligned(E, dt)) || (P && !elem_aligned(P, dt)))
    return fail(SN_ERR_ALIGN, "E or P not aligned to its element size");
  const sn::ProjLayout PL = sn::proj_layout(k, vocab, n_pos);
  if (PL.total == 0) return ok();
  if (!proj) return fail(SN_ERR_NULL, "proj is NULL");
  if (reinterpret_cast<uintptr_t>(proj) & 255)
    return fail(SN_ERR_ALIGN, "proj must be 256-byte aligned");
  if (proj_bytes < PL.total)
    return fail(SN_ERR_WORKSPACE, "proj has %zu bytes, needs %zu", proj_bytes, PL.total);
  const size_t es = elem_size(dt);
  const sn::PackLayout L = sn::pack_layout(d, k, dt);
  Span out;
  out.lo = reinterpret_cast<uintptr_t>(proj);
  out.hi = out.lo + PL.total;
  Span b;
  b.lo = reinterpret_cast<uintptr_t>(basis);
  b.hi = b.lo + L.total;
  if (overlap(out, b) || overlap(out, span(E, vocab, d, lde, es)) ||
      overlap(out, span(P, n_pos, d, ldp, es)))
    return fail(SN_ERR_ALIAS, "proj overlaps the basis, E or P");
  hipStream_t s = static_cast<hipStream_t>(stream);
  char *base = static_cast<char *>(proj);
  const struct {
    const void *t;
    int64_t rows, ld;
    size_t off;
  } parts[2] = {{E, vocab, lde, PL.off_eu}, {P, n_pos, ldp, PL.off_pu}};
  for (const auto &pt : parts) {
    if (pt.rows == 0) continue;
    float *o = reinterpret_cast<float *>(base + pt.off);
    hipError_t e = sn::stream_mfma_ok(L, pt.t, pt.ld)
                       ? sn::launch_table_project_mfma(L, basis, pt.t, pt.rows, pt.ld, o, PL.kp, s)
                       : sn::launch_table_project_generic(L, basis, pt.t, pt.rows, pt.ld, o,
                                                          PL.kp, s);
    if (e != hipSuccess) return hip_status(e, "sn_embed_project launch");
  }
  return ok();
}

int32_t sn_compress_projected(const void *basis, int64_t d, int64_t k, int32_t dt, const void *X,
                              int64_t N, int64_t ldx, const int32_t *tok, const int32_t *pos,
                              int64_t seq_len, const void *proj, int64_t vocab, int64_t n_pos,
                              void *C, int64_t ldc, int32_t *err_flag, sn_stream stream) {
  int32_t st = check_basis(basis, d, k, dt);
  if (st) return st;
  if (N < 0 || N >= kMaxDim) return fail(SN_ERR_SHAPE, "N = %lld out of range", (long long)N);
  if (ldx < d || ldx >= kMaxDim) return fail(SN_ERR_SHAPE, "ldx must be >= d");
  if (ldc < k || ldc >= kMaxDim) return fail(SN_ERR_SHAPE, "ldc must be >= k");
  if (vocab < 0 || vocab >= kMaxDim) return fail(SN_ERR_SHAPE, "vocab out of range");
  if (n_pos < 0 || n_pos >= kMaxDim) return fail(SN_ERR_SHAPE, "n_pos out of range");
  if ((vocab > 0 || n_pos > 0) && !proj) return fail(SN_ERR_NULL, "proj is NULL");
  if (proj && (reinterpret_cast<uintptr_t>(proj) & 255))
    return fail(SN_ERR_ALIGN, "proj must be 256-byte aligned");
  if (n_pos > 0 && !pos && (seq_len < 1 || seq_len > n_pos))
    return fail(SN_ERR_SHAPE, "pos is NULL: need 1 <= seq_len <= n_pos (seq_len = %lld)",
                (long long)seq_len);
  if ((tok && (reinterpret_cast<uintptr_t>(tok) & 3)) ||
      (pos && (reinterpret_cast<uintptr_t>(pos) & 3)))
    return fail(SN_ERR_ALIGN, "tok / pos not 4-byte aligned");
  if (N == 0) return ok();
  if (vocab > 0 && !tok) return fail(SN_ERR_NULL, "tok is NULL but vocab > 0");
  if (!X || !C) return fail(SN_ERR_NULL, "X or C is NULL");
  if (!elem_aligned(X, dt) || !elem_aligned(C, dt))
    return fail(SN_ERR_ALIGN, "X or C not aligned to its element size");
  const size_t es = elem_size(dt);
  const sn::PackLayout L = sn::pack_layout(d, k, dt);
  const sn::ProjLayout PL = sn::proj_layout(k, vocab, n_pos);
  const Span out = span(C, N, k, ldc, es);
  Span b;
  b.lo = reinterpret_cast<uintptr_t>(basis);
  b.hi = b.lo + L.total;
  Span pj;
  if (proj) {
    pj.lo = reinterpret_cast<uintptr_t>(proj);
    pj.hi = pj.lo + PL.total;
  }
  if (overlap(out, b) || overlap(out, pj) || overlap(out, span(X, N, d, ldx, es)) ||
      (vocab > 0 && overlap(out, span(tok, 1, N, N, 4))) ||
      (n_pos > 0 && pos && overlap(out, span(pos, 1, N, N, 4))))
    return fail(SN_ERR_ALIAS, "C overlaps an input");
  const char *pb = static_cast<const char *>(proj);
  sn::ProjArgs pa{};
  pa.tok = vocab > 0 ? tok : nullptr;
  pa.eu = vocab > 0 ? reinterpret_cast<const float *>(pb + PL.off_eu) : nullptr;
  pa.vocab = vocab;
  pa.pos = n_pos > 0 ? pos : nullptr;
  pa.pu = n_pos > 0 ? reinterpret_cast<const float *>(pb + PL.off_pu) : nullptr;
  pa.n_pos = n_pos;
  pa.seq_len = (n_pos > 0 && !pos) ? seq_len : 1;
  pa.kp = PL.kp;
  pa.err_flag = err_flag;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (sn::stream_mfma_ok(L, X, ldx))
    return hip_status(sn::launch_compress_projected_mfma(L, basis, X, N, ldx, pa, C, ldc, s),
                      "sn_compress_projected launch");
  return hip_status(sn::launch_compress_projected_generic(L, basis, X, N, ldx, pa, C, ldc, s),
                    "sn_compress_projected launch");
}

size_t sn_project_weights_workspace_bytes(int64_t d, int64_t k, int32_t dt, int64_t m) {
  if (!dtype_ok(dt) || d < 1 || d >= kMaxDim || k < 1 || k > d || k > SN_MAX_K || m < 0 ||
      m >= kMaxDim)
    return 0;
  const sn::PackLayout L = sn::pack_layout(d, k, dt);
  size_t a = sn::project_workspace_generic(d, k, m);
  size_t b = L.mfma ? sn::project_workspace_mfma(d, k, m) : 0;
  return sn::align256(a > b ? a : b);
}

int32_t sn_project_weights(const void *basis, int64_t d, int64_t k, int32_t dt, void *W,
                           int64_t m, int64_t ldw, void *workspace, size_t workspace_bytes,
                           sn_stream stream) {
  int32_t st = sn::project_args_check(basis, d, k, dt, W, m, ldw);
  if (st) return st;
  if (m == 0) return ok();
  if (!workspace) return fail(SN_ERR_NULL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) & 255)
    return fail(SN_ERR_ALIGN, "workspace must be 256-byte aligned");
  const size_t need = sn_project_weights_workspace_bytes(d, k, dt, m);
  if (workspace_bytes < need)
    return fail(SN_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
  const sn::PackLayout L = sn::pack_layout(d, k, dt);
  Span w = span(W, d, m, ldw, elem_size(dt));
  Span ws;
  ws.lo = reinterpret_cast<uintptr_t>(workspace);
  ws.hi = ws.lo + need;
  Span b;
  b.lo = reinterpret_cast<uintptr_t>(basis);
  b.hi = b.lo + L.total;
  if (overlap(w, ws) || overlap(w, b) || overlap(ws, b))
    return fail(SN_ERR_ALIAS, "W, workspace and basis must not overlap");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (L.mfma && sn::project_mfma_ok(L, W, m, ldw))
    return hip_status(sn::launch_project_mfma(L, basis, W, m, ldw, workspace, s),
                      "sn_project_weights launch");
  return hip_status(sn::launch_project_generic(L, basis, W, m, ldw, workspace, s),
                    "sn_project_weights launch");
}

size_t sn_grassmann_state_bytes(int64_t d, int64_t k) {
  if (d < 1 || d >= kMaxDim || k < 1 || k > d || k > sn::kGrassMaxK) return 0;
  return sn::grass_state_bytes(d, k);
}

size_t sn_grassmann_workspace_bytes(int64_t d, int64_t k, int32_t dt, int64_t N) {
  if (!dtype_ok(dt) || d < 1 || d >= kMaxDim || k < 1 || k > d || k > sn::kGrassMaxK || N < 0 ||
      N >= kMaxDim)
    return 0;
  return sn::grass_workspace_bytes(sn::pack_layout(d, k, dt), N);
}

int32_t sn_grassmann_reset(void *state, int64_t d, int64_t k, sn_stream stream) {
  if (d < 1 || d >= kMaxDim || k < 1 || k > d) return fail(SN_ERR_SHAPE, "need 1 <= k <= d");
  int32_t st = check_state(state, d, k);
  if (st) return st;
  return hip_status(sn::launch_grass_reset(state, d, k, static_cast<hipStream_t>(stream)),
                    "sn_grassmann_reset launch");
}

int32_t sn_grassmann_accumulate(const void *basis, int64_t d, int64_t k, int32_t dt, const void *G,
                                int64_t N, int64_t ldg, void *Cg, int64_t ldc, int32_t with_su,
                                void *state, void *workspace, size_t workspace_bytes,
                                sn_stream stream) {
  int32_t st = check_basis(basis, d, k, dt);
  if (st) return st;
  if ((st = check_state(state, d, k))) return st;
  if (N < 0 || N >= kMaxDim) return fail(SN_ERR_SHAPE, "N = %lld out of range", (long long)N);
  if (ldg < d || ldg >= kMaxDim) return fail(SN_ERR_SHAPE, "ldg must be >= d");
  if (Cg && (ldc < k || ldc >= kMaxDim)) return fail(SN_ERR_SHAPE, "ldc must be >= k");
  if (N == 0) return ok();
  if (!G) return fail(SN_ERR_NULL, "G is NULL");
  if (!elem_aligned(G, dt) || (Cg && !elem_aligned(Cg, dt)))
    return fail(SN_ERR_ALIGN, "G or Cg not aligned to its element size");
  const size_t need = sn_grassmann_workspace_bytes(d, k, dt, N);
  if ((st = check_workspace(workspace, workspace_bytes, need))) return st;
  const size_t es = elem_size(dt);
  const sn::PackLayout L = sn::pack_layout(d, k, dt);
  const Span g = span(G, N, d, ldg, es), c = span(Cg, N, k, ldc, es);
  const Span b = bytes_span(basis, L.total), sb = bytes_span(state, sn::grass_state_bytes(d, k));
  const Span w = bytes_span(workspace, need);
  if (overlap(c, g) || overlap(c, b) || overlap(c, sb) || overlap(c, w))
    return fail(SN_ERR_ALIAS, "Cg overlaps an input, the state or the workspace");
  if (overlap(sb, g) || overlap(sb, b) || overlap(sb, w))
    return fail(SN_ERR_ALIAS, "state overlaps G, the basis or the workspace");
  if (overlap(w, g) || overlap(w, b))
    return fail(SN_ERR_ALIAS, "workspace overlaps G or the basis");
  return hip_status(sn::launch_grass_accumulate(L, basis, G, N, ldg, Cg, ldc, with_su != 0, state,
                                                workspace, static_cast<hipStream_t>(stream)),
                    "sn_grassmann_accumulate launch");
}

int32_t sn_grassmann_step(const void *basis, int64_t d, int64_t k, int32_t dt, const void *state,
                          double eta, void *U_new, int64_t ldu, int32_t out_dt, void *workspace,
                          size_t workspace_bytes, int32_t *err_flag, sn_stream stream) {
  int32_t st = check_basis(basis, d, k, dt);
  if (st) return st;
  if ((st = check_state(state, d, k))) return st;
  if (!dtype_ok(out_dt)) return fail(SN_ERR_DTYPE, "unknown out_dt %d", out_dt);
  if (!(eta >= 0.0) || eta > 1e300) return fail(SN_ERR_SHAPE, "eta must be finite and >= 0");
  if (!U_new) return fail(SN_ERR_NULL, "U_new is NULL");
  if (ldu < k || ldu >= kMaxDim) return fail(SN_ERR_SHAPE, "ldu must be >= k");
  if (!elem_aligned(U_new, out_dt)) return fail(SN_ERR_ALIGN, "U_new not aligned");
  if (err_flag && (reinterpret_cast<uintptr_t>(err_flag) & 3))
    return fail(SN_ERR_ALIGN, "err_flag not 4-byte aligned");
  const size_t need = sn_grassmann_workspace_bytes(d, k, dt, 0);
  if ((st = check_workspace(workspace, workspace_bytes, need))) return st;
  const sn::PackLayout L = sn::pack_layout(d, k, dt);
  const Span u = span(U_new, d, k, ldu, elem_size(out_dt));
  const Span b = bytes_span(basis, L.total), sb = bytes_span(state, sn::grass_state_bytes(d, k));
  const Span w = bytes_span(workspace, need);
  if (overlap(u, b) || overlap(u, sb) || overlap(u, w))
    return fail(SN_ERR_ALIAS, "U_new overlaps the basis, the state or the workspace");
  if (overlap(w, b) || overlap(w, sb))
    return fail(SN_ERR_ALIAS, "workspace overlaps the basis or the state");
  return hip_status(sn::launch_grass_step(L, basis, state, eta, U_new, ldu, out_dt, workspace,
                                          err_flag, static_cast<hipStream_t>(stream)),
                    "sn_grassmann_step launch");
}

size_t sn_embed_lowrank_workspace_bytes(int64_t d, int64_t k, int32_t dt, int64_t N,
                                        int64_t vocab) {
  if (!dtype_ok(dt) || d < 1 || d >= kMaxDim || k < 1 || k > d || k > SN_MAX_K || N < 0 ||
      N >= kMaxDim || vocab < 1 || vocab >= kMaxDim)
    return 0;
  return sn::embed_workspace_bytes(k, dt, N, vocab);
}

int32_t sn_embed_lowrank_forward(const void *basis, int64_t d, int64_t k, int32_t dt,
                                 const void *CS, int64_t vocab, int64_t ldcs, const int32_t *tok,
                                 const void *E, int64_t lde, const int32_t *pos, const void *P,
                                 int64_t n_pos, int64_t ldp, int64_t seq_len, void *X0,
                                 int64_t N, int64_t ldx, int32_t *err_flag, void *workspace,
                                 size_t workspace_bytes, sn_stream stream) {
  int32_t st = check_basis(basis, d, k, dt);
  if (st) return st;
  if (N < 0 || N >= kMaxDim) return fail(SN_ERR_SHAPE, "N out of range");
  if (vocab < 1 || vocab >= kMaxDim) return fail(SN_ERR_SHAPE, "vocab out of range");
  if (ldcs < k || ldcs >= kMaxDim) return fail(SN_ERR_SHAPE, "ldcs must be >= k");
  if (ldx < d || ldx >= kMaxDim) return fail(SN_ERR_SHAPE, "ldx must be >= d");
  if ((st = check_ids(N, d, dt, tok, E, vocab, lde, pos, P, n_pos, ldp, seq_len))) return st;
  if (N == 0) return ok();
  if (!CS || !tok || !X0) return fail(SN_ERR_NULL, "CS, tok and X0 are required");
  if (!elem_aligned(CS, dt) || !elem_aligned(X0, dt) || (reinterpret_cast<uintptr_t>(tok) & 3))
    return fail(SN_ERR_ALIGN, "CS, X0 or tok misaligned");
  const size_t need = sn_embed_lowrank_workspace_bytes(d, k, dt, N, vocab);
  if ((st = check_workspace(workspace, workspace_bytes, need))) return st;
  const size_t es = elem_size(dt);
  const sn::PackLayout L = sn::pack_layout(d, k, dt);
  const Span x = span(X0, N, d, ldx, es), w = bytes_span(workspace, need);
  if ((st = check_out_alias(x, basis, L.total, span(CS, vocab, k, ldcs, es), N, tok, E, vocab,
                            lde, pos, P, n_pos, ldp, d, es)))
    return st;
  if (overlap(x, span(tok, 1, N, N, 4)) || overlap(x, w) || overlap(w, span(CS, vocab, k, ldcs, es)) ||
      overlap(w, span(tok, 1, N, N, 4)) || overlap(w, bytes_span(basis, L.total)) ||
      (E && overlap(w, span(E, vocab, d, lde, es))) || (P && overlap(w, span(P, n_pos, d, ldp, es))))
    return fail(SN_ERR_ALIAS, "X0 or the workspace overlaps an input");
  const sn::IdArgs ids = make_ids(tok, E, vocab, lde, pos, P, n_pos, ldp, seq_len, err_flag);
  return hip_status(sn::launch_embed_forward(L, basis, CS, vocab, ldcs, tok, ids, N, X0, ldx,
                                             workspace, static_cast<hipStream_t>(stream)),
                    "sn_embed_lowrank_forward launch");
}

int32_t sn_embed_lowrank_backward(const void *basis, int64_t d, int64_t k, int32_t dt,
                                  const void *dX0, int64_t N, int64_t ldg, const int32_t *tok,
                                  int64_t vocab, float *gCS, int64_t ldgc, int32_t *err_flag,
                                  void *workspace, size_t workspace_bytes, sn_stream stream) {
  int32_t st = check_basis(basis, d, k, dt);
  if (st) return st;
  if (N < 0 || N >= kMaxDim) return fail(SN_ERR_SHAPE, "N out of range");
  if (vocab < 1 || vocab >= kMaxDim) return fail(SN_ERR_SHAPE, "vocab out of range");
  if (ldg < d || ldg >= kMaxDim) return fail(SN_ERR_SHAPE, "ldg must be >= d");
  if (ldgc < k || ldgc >= kMaxDim) return fail(SN_ERR_SHAPE, "ldgc must be >= k");
  if (vocab >= (int64_t(1) << 21))
    return fail(SN_ERR_UNSUPPORTED, "the gradient scatter sorts ids below 2^21 (vocab = %lld)",
                (long long)vocab);
  if (N == 0) return ok();
  if (!dX0 || !tok || !gCS) return fail(SN_ERR_NULL, "dX0, tok and gCS are required");
  if (!elem_aligned(dX0, dt) || !elem_aligned(gCS, SN_F32) ||
      (reinterpret_cast<uintptr_t>(tok) & 3))
    return fail(SN_ERR_ALIGN, "dX0, gCS or tok misaligned");
  const size_t need = sn_embed_lowrank_workspace_bytes(d, k, dt, N, vocab);
  if ((st = check_workspace(workspace, workspace_bytes, need))) return st;
  const sn::PackLayout L = sn::pack_layout(d, k, dt);
  const Span g = span(gCS, vocab, k, ldgc, 4), w = bytes_span(workspace, need);
  const Span x = span(dX0, N, d, ldg, elem_size(dt)), t = span(tok, 1, N, N, 4);
  const Span b = bytes_span(basis, L.total);
  if (overlap(g, x) || overlap(g, t) || overlap(g, w) || overlap(g, b) || overlap(w, x) ||
      overlap(w, t) || overlap(w, b))
    return fail(SN_ERR_ALIAS, "gCS, the workspace and the inputs must not overlap");
  return hip_status(sn::launch_embed_backward(L, basis, dX0, N, ldg, tok, vocab, gCS, ldgc,
                                              err_flag, workspace,
                                              static_cast<hipStream_t>(stream)),
                    "sn_embed_lowrank_backward launch");
}

size_t sn_adamw_workspace_bytes(int64_t rows, int64_t cols) {
  if (rows < 0 || rows >= kMaxDim || cols < 0 || cols >= kMaxDim) return 0;
  return sn::adamw_workspace_bytes(rows, cols);
}

int32_t sn_adamw_step(void *W, int64_t ldw, const void *G, int64_t ldg, int32_t dt, float *M,
                      float *V, int64_t ldm, int64_t rows, int64_t cols, int64_t t, double lr,
                      double beta1, double beta2, double eps, double weight_decay,
                      int32_t subspace, void *workspace, size_t workspace_bytes,
                      sn_stream stream) {
  if (!dtype_ok(dt)) return fail(SN_ERR_DTYPE, "unknown dtype %d", dt);
  if (rows < 0 || rows >= kMaxDim || cols < 0 || cols >= kMaxDim)
    return fail(SN_ERR_SHAPE, "rows / cols out of range");
  if (t < 1) return fail(SN_ERR_SHAPE, "t counts steps from 1 (t = %lld)", (long long)t);
  if (!(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0))
    return fail(SN_ERR_SHAPE, "betas must lie in [0, 1)");
  if (!(eps >= 0.0 && eps <= 1e30) || !(lr >= 0.0 && lr <= 1e30) ||
      !(weight_decay >= 0.0 && weight_decay <= 1e30))
    return fail(SN_ERR_SHAPE, "lr, eps and weight_decay must be finite and >= 0");
  if (rows == 0 || cols == 0) return ok();
  if (ldw < cols || ldg < cols || ldm < cols || ldw >= kMaxDim || ldg >= kMaxDim ||
      ldm >= kMaxDim)
    return fail(SN_ERR_SHAPE, "row strides must be >= cols");
  if (!W || !G || !M || !V) return fail(SN_ERR_NULL, "W, G, M and V are required");
  if (!elem_aligned(W, dt) || !elem_aligned(G, dt) || !elem_aligned(M, SN_F32) ||
      !elem_aligned(V, SN_F32))
    return fail(SN_ERR_ALIGN, "W, G, M or V not aligned to its element size");
  int32_t st;
  const size_t need = subspace ? sn_adamw_workspace_bytes(rows, cols) : 0;
  if (subspace && (st = check_workspace(workspace, workspace_bytes, need))) return st;
  const size_t es = elem_size(dt);
  const Span w = span(W, rows, cols, ldw, es), g = span(G, rows, cols, ldg, es);
  const Span m = span(M, rows, cols, ldm, 4), v = span(V, rows, cols, ldm, 4);
  const Span ws = subspace ? bytes_span(workspace, need) : Span{};
  const Span all[5] = {w, g, m, v, ws};
  for (int i = 0; i < 5; ++i)
    for (int j = i + 1; j < 5; ++j)
      if (overlap(all[i], all[j]))
        return fail(SN_ERR_ALIAS, "W, G, M, V and the workspace must not overlap");
  return hip_status(sn::launch_adamw(dt, W, ldw, G, ldg, M, V, ldm, rows, cols, t, lr, beta1,
                                     beta2, eps, weight_decay, subspace != 0, workspace,
                                     static_cast<hipStream_t>(stream)),
                    "sn_adamw_step launch");
}

namespace {

// The segmented (one set of launches) form applies when every matrix meets
// the MFMA path's conditions with a width that is a multiple of 256.
bool multi_segmented(const sn::PackLayout &L, int32_t count, void *const *W, const int64_t *m,
                     const int64_t *ldw) {
  if (!L.mfma || L.ks2 == 0 || count < 1 || count > sn::kMaxSeg) return false;
  for (int32_t i = 0; i < count; ++i)
    if (m[i] % 256 != 0 || !sn::project_mfma_ok(L, W[i], m[i], ldw[i])) return false;
  return true;
}

}  // namespace

size_t sn_project_weights_multi_workspace_bytes(int64_t d, int64_t k, int32_t dt, int32_t count,
                                                const int64_t *m) {
  if (!dtype_ok(dt) || d < 1 || d >= kMaxDim || k < 1 || k > d || k > SN_MAX_K || count < 0 ||
      count > SN_PROJECT_MAX_MATRICES || (count > 0 && !m))
    return 0;
  size_t best = 0;
  int64_t total = 0;
  for (int32_t i = 0; i < count; ++i) {
    if (m[i] < 0 || m[i] >= kMaxDim) return 0;
    const size_t one = sn_project_weights_workspace_bytes(d, k, dt, m[i]);
    best = one > best ? one : best;
    total += m[i];
  }
  if (total >= kMaxDim) return 0;
  const sn::PackLayout L = sn::pack_layout(d, k, dt);
  if (L.mfma && total > 0) {
    const size_t seg = sn::align256(sn::project_workspace_mfma(d, k, total));
    best = seg > best ? seg : best;
  }
  return best;
}

int32_t sn_project_weights_multi(const void *basis, int64_t d, int64_t k, int32_t dt, int32_t count,
                                 void *const *W, const int64_t *m, const int64_t *ldw,
                                 void *workspace, size_t workspace_bytes, sn_stream stream) {
  int32_t st = check_basis(basis, d, k, dt);
  if (st) return st;
  if (count < 0 || count > SN_PROJECT_MAX_MATRICES)
    return fail(SN_ERR_SHAPE, "count must lie in [0, %d]", SN_PROJECT_MAX_MATRICES);
  if (count == 0) return ok();
  if (!W || !m || !ldw) return fail(SN_ERR_NULL, "W, m and ldw arrays are required");
  int64_t total = 0;
  for (int32_t i = 0; i < count; ++i) {
    if (m[i] < 0 || m[i] >= kMaxDim) return fail(SN_ERR_SHAPE, "m[%d] out of range", i);
    if (ldw[i] < m[i] || ldw[i] >= kMaxDim) return fail(SN_ERR_SHAPE, "ldw[%d] must be >= m[%d]", i, i);
    if (m[i] > 0 && !W[i]) return fail(SN_ERR_NULL, "W[%d] is NULL", i);
    if (m[i] > 0 && !elem_aligned(W[i], dt)) return fail(SN_ERR_ALIGN, "W[%d] misaligned", i);
    total += m[i];
  }
  if (total >= kMaxDim) return fail(SN_ERR_SHAPE, "total width out of range");
  if (total == 0) return ok();
  if (!workspace) return fail(SN_ERR_NULL, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) & 255)
    return fail(SN_ERR_ALIGN, "workspace must be 256-byte aligned");
  const size_t need = sn_project_weights_multi_workspace_bytes(d, k, dt, count, m);
  if (workspace_bytes < need)
    return fail(SN_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
  const sn::PackLayout L = sn::pack_layout(d, k, dt);
  const size_t es = elem_size(dt);
  const Span ws = bytes_span(workspace, need), b = bytes_span(basis, L.total);
  if (overlap(ws, b)) return fail(SN_ERR_ALIAS, "workspace overlaps the basis");
  for (int32_t i = 0; i < count; ++i) {
    const Span wi = span(W[i], d, m[i], ldw[i], es);
    if (overlap(wi, ws) || overlap(wi, b))
      return fail(SN_ERR_ALIAS, "W[%d] overlaps the workspace or the basis", i);
    for (int32_t j = 0; j < i; ++j)
      if (overlap(wi, span(W[j], d, m[j], ldw[j], es)))
        return fail(SN_ERR_ALIAS, "W[%d] overlaps W[%d]", i, j);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (multi_segmented(L, count, W, m, ldw)) {
    sn::ColSegs cs;
    cs.n = 0;
    int64_t c0 = 0;
    for (int32_t i = 0; i < count; ++i) {
      if (m[i] == 0) continue;
      cs.c0[cs.n] = c0;
      cs.base[cs.n] = W[i];
      cs.ld[cs.n] = ldw[i];
      ++cs.n;
      c0 += m[i];
    }
    cs.c0[cs.n] = c0;
    return hip_status(sn::launch_project_mfma_segs(L, basis, cs, workspace, s),
                      "sn_project_weights_multi launch");
  }
  for (int32_t i = 0; i < count; ++i) {  // one after another, sharing the workspace
    if (m[i] == 0) continue;
    if ((st = sn_project_weights(basis, d, k, dt, W[i], m[i], ldw[i], workspace, workspace_bytes,
                                 stream)))
      return st;
  }
  return ok();
}

const char *sn_status_string(int32_t status) {
  switch (status) {
    case SN_OK: return "SN_OK";
    case SN_ERR_NULL: return "SN_ERR_NULL";
    case SN_ERR_SHAPE: return "SN_ERR_SHAPE";
    case SN_ERR_DTYPE: return "SN_ERR_DTYPE";
    case SN_ERR_ALIGN: return "SN_ERR_ALIGN";
    case SN_ERR_ALIAS: return "SN_ERR_ALIAS";
    case SN_ERR_INDEX: return "SN_ERR_INDEX";
    case SN_ERR_HIP: return "SN_ERR_HIP";
    case SN_ERR_UNSUPPORTED: return "SN_ERR_UNSUPPORTED";
    case SN_ERR_WORKSPACE: return "SN_ERR_WORKSPACE";
    default: return "SN_ERR_UNKNOWN";
  }
}

const char *sn_last_error(void) { return g_err; }

const char *sn_version(void) { return "0.1.0 gfx950"; }

}  // extern "C"
