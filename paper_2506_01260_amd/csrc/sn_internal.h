// Host-side internals of the codec library: the packed-basis layout and the
// kernel launchers the C ABI dispatches to.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sn {

constexpr int kMaxK = 256;      // SN_MAX_K
constexpr int kMfmaMaxKT = 8;   // MFMA path: k <= 128 (8 column tiles of 16)

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// Packed basis (one device buffer, sections 256-byte aligned):
//
//  f32   U as float32, d x k, row stride k.  Read by the generic kernels.
//  kfrag (bf16 and d % 32 == 0 and k <= 128 only) U in the MFMA operand layout
//        of a contraction over d (compress, projection pass 1): 1 KiB blocks
//        indexed [s][t], s = d/32 row steps, t = ceil(k/16) column tiles;
//        lane l = 16 g + n of block (s, t) holds the 8 bf16
//        U[32 s + 8 g + e, 16 t + n], e = 0..7 (0 past column k).
//  rfrag (same condition) U in the MFMA operand layout of a contraction over k
//        (decompress, projection pass 2): 1 KiB blocks indexed [p][h][q],
//        p = d/32 row groups, h = 0..1, q = ceil(k/32) k-steps; lane
//        l = 16 g + m holds the 8 bf16 U[32 p + 8 (m/4) + 4 h + m%4, 32 q + 8 g + e].
//        The row order puts 8 consecutive d-rows of one token in one lane of
//        the MFMA result, so decompress stores 16 bytes per lane.
//  uu    (same condition and k <= 64) [U | U] as bf16, d x 32 ceil(2k/32),
//        columns past 2k zero: the coefficients of the weight projection's
//        second contraction written as a decompress.
//  gram  (every basis) U^T U - I as float64, kp x kp with kp = 16 ceil(k/16)
//        (zero outside k x k): the stored basis's departure from
//        orthonormality, used by the off-subspace loss.
struct PackLayout {
  int64_t d = 0, k = 0;
  int dt = 0;
  bool mfma = false;
  int kt = 0;   // ceil(k/16)
  int ks = 0;   // ceil(k/32)
  int ks2 = 0;  // ceil(2k/32) when the uu section exists, else 0
  size_t off_f32 = 0, off_kfrag = 0, off_rfrag = 0, off_uu = 0, off_gram = 0, total = 0;
};

PackLayout pack_layout(int64_t d, int64_t k, int dt);

// A matrix given as column segments side by side, each with its own base
// pointer and row stride: segment s holds global columns [c0[s], c0[s+1]).
// The decompress and projection kernels read and write it as one matrix, so
// several weights of the same d are projected by one set of launches.
constexpr int kMaxSeg = 16;  // SN_PROJECT_MAX_MATRICES
struct ColSegs {
  int n = 1;
  int64_t c0[kMaxSeg + 1] = {};
  void *base[kMaxSeg] = {};
  int64_t ld[kMaxSeg] = {};
};
inline ColSegs one_seg(const void *p, int64_t cols, int64_t ld) {
  ColSegs c;
  c.n = 1;
  c.c0[0] = 0;
  c.c0[1] = cols;
  c.base[0] = const_cast<void *>(p);
  c.ld[0] = ld;
  return c;
}

// ---- launchers (arguments already validated; N > 0) ----------------------
struct IdArgs {
  const int32_t *tok;
  const void *E;
  int64_t vocab, lde;
  const int32_t *pos;
  const void *P;
  int64_t n_pos, ldp, seq_len;
  int32_t *err_flag;
};

hipError_t launch_pack(const PackLayout &L, const void *U, int64_t ldu, void *packed,
                       hipStream_t s);

hipError_t launch_compress_generic(const PackLayout &L, const void *packed, const void *X,
                                   int64_t N, int64_t ldx, const IdArgs &ids, void *C,
                                   int64_t ldc, hipStream_t s);
hipError_t launch_decompress_generic(const PackLayout &L, const void *packed, const void *C,
                                     int64_t N, int64_t ldc, const IdArgs &ids, void *X,
                                     int64_t ldx, hipStream_t s);

size_t project_workspace_generic(int64_t d, int64_t k, int64_t m);
hipError_t launch_project_generic(const PackLayout &L, const void *packed, void *W, int64_t m,
                                  int64_t ldw, void *ws, hipStream_t s);

// MFMA paths (bf16, L.mfma).  Return hipErrorNotSupported if the arguments do
// not fit the fast path; the caller then uses the generic kernels.
bool compress_mfma_ok(const PackLayout &L, const void *X, int64_t ldx, const IdArgs &ids);
hipError_t launch_compress_mfma(const PackLayout &L, const void *packed, const void *X,
                                int64_t N, int64_t ldx, const IdArgs &ids, void *C, int64_t ldc,
                                hipStream_t s);
bool decompress_mfma_ok(const PackLayout &L, void *X, int64_t ldx, const IdArgs &ids);
hipError_t launch_decompress_mfma(const PackLayout &L, const void *packed, const void *C,
                                  int64_t N, int64_t ldc, const IdArgs &ids, void *X,
                                  int64_t ldx, hipStream_t s);
// the same with X given as column segments (each width a multiple of 256)
hipError_t launch_decompress_mfma_segs(const PackLayout &L, const void *packed, const void *C,
                                       int64_t N, int64_t ldc, const IdArgs &ids,
                                       const ColSegs &X, hipStream_t s);

// Projected tables: T_fixed U (vocab rows) then P U (n_pos rows), fp32, row
// stride kp = 16 * ceil(k / 16) (columns k..kp-1 are zero), the P U section at
// a 256-byte aligned offset.
struct ProjLayout {
  int64_t kp = 0;
  size_t off_eu = 0, off_pu = 0, total = 0;
};
ProjLayout proj_layout(int64_t k, int64_t vocab, int64_t n_pos);

// Ids and projected rows of a compress against projected tables; eu / pu
// NULL = no token / positional term.
struct ProjArgs {
  const int32_t *tok;
  const float *eu;
  int64_t vocab;
  const int32_t *pos;
  const float *pu;
  int64_t n_pos, seq_len;
  int64_t kp;
  int32_t *err_flag;
};

bool stream_mfma_ok(const PackLayout &L, const void *X, int64_t ldx);
// rows x d table -> rows x kp fp32 (T U), MFMA path
hipError_t launch_table_project_mfma(const PackLayout &L, const void *packed, const void *T,
                                     int64_t rows, int64_t ldt, float *out, int64_t kp,
                                     hipStream_t s);
hipError_t launch_compress_projected_mfma(const PackLayout &L, const void *packed, const void *X,
                                          int64_t N, int64_t ldx, const ProjArgs &pa, void *C,
                                          int64_t ldc, hipStream_t s);
hipError_t launch_table_project_generic(const PackLayout &L, const void *packed, const void *T,
                                        int64_t rows, int64_t ldt, float *out, int64_t kp,
                                        hipStream_t s);
hipError_t launch_compress_projected_generic(const PackLayout &L, const void *packed,
                                             const void *X, int64_t N, int64_t ldx,
                                             const ProjArgs &pa, void *C, int64_t ldc,
                                             hipStream_t s);

size_t project_workspace_mfma(int64_t d, int64_t k, int64_t m);

// ---- subspace update (Sec. 4.5) ---------------------------------------------
// The compress epilogue that feeds the subspace update: each workgroup's sum
// of the rows' loss terms |g|^2 - |c|^2 + c D c^T (D = U^T U - I, kp x kp
// float64, kp = 16 ceil(k/16)) into part[workgroup], and with frag the token
// contraction's operand (C split into bf16 hi + lo in the kfrag layout:
// nparts operands of ktb column tiles and npad rows).
struct GrassOut {
  const double *dgram = nullptr;
  double *part = nullptr;
  uint16_t *frag = nullptr;  // bf16 bits
  int nparts = 0, ktb = 0;
  int64_t npad = 0;
};
hipError_t launch_grass_compress_mfma(const PackLayout &L, const void *packed, const void *G,
                                      int64_t N, int64_t ldg, const GrassOut &go, void *Cwire,
                                      int64_t ldc, hipStream_t s);
// Workgroups (loss partials) of that compress for N rows, and 32-row steps
// of the operand it writes.
int64_t grass_compress_groups(const PackLayout &L, int64_t N, int64_t *steps);
// Tp[split][i][j] = sum over the split's token rows n of F[n, j] G[n, i]
// (F in the kfrag layout with ktb column tiles and npad rows, zero past N).
hipError_t launch_grass_tokens_mfma(const void *frag, int ktb, int64_t npad, const void *G,
                                    int64_t N, int64_t ldg, int64_t d, int64_t rows, int ds,
                                    int64_t m_pad, float *Tp, hipStream_t s);

constexpr size_t kGrassStateHead = 256;  // bytes before Y in the accumulator state
constexpr int kGrassMaxK = 128;          // largest k of the subspace update
size_t grass_state_bytes(int64_t d, int64_t k);
size_t grass_workspace_bytes(const PackLayout &L, int64_t N);
bool grass_mfma_ok(const PackLayout &L, const void *G, int64_t ldg);
hipError_t launch_grass_reset(void *state, int64_t d, int64_t k, hipStream_t s);
hipError_t launch_grass_accumulate(const PackLayout &L, const void *packed, const void *G,
                                   int64_t N, int64_t ldg, void *Cwire, int64_t ldc, bool with_su,
                                   void *state, void *ws, hipStream_t s);
// ---- low-rank token table (Sec. 4.3.1) -------------------------------------------
size_t embed_workspace_bytes(int64_t k, int dt, int64_t N, int64_t vocab);
hipError_t launch_embed_forward(const PackLayout &L, const void *packed, const void *CS,
                                int64_t vocab, int64_t ldcs, const int32_t *tok,
                                const IdArgs &ids, int64_t N, void *X0, int64_t ldx, void *ws,
                                hipStream_t s);
hipError_t launch_embed_backward(const PackLayout &L, const void *packed, const void *dX0,
                                 int64_t N, int64_t ldg, const int32_t *tok, int64_t vocab,
                                 float *gCS, int64_t ldgc, int32_t *err_flag, void *ws,
                                 hipStream_t s);

// ---- modified AdamW (Sec. 5) ---------------------------------------------------
size_t adamw_workspace_bytes(int64_t rows, int64_t cols);
hipError_t launch_adamw(int dt, void *W, int64_t ldw, const void *G, int64_t ldg, float *M,
                        float *V, int64_t ldm, int64_t rows, int64_t cols, int64_t t, double lr,
                        double beta1, double beta2, double eps, double wd, bool subspace,
                        void *ws, hipStream_t s);

hipError_t launch_grass_step(const PackLayout &L, const void *packed, const void *state,
                             double eta, void *Unew, int64_t ldu, int out_dt, void *ws,
                             int32_t *err_flag, hipStream_t s);
bool project_mfma_ok(const PackLayout &L, const void *W, int64_t m, int64_t ldw);
// W <- U (U^T W) for the matrix of column segments W (every width a multiple
// of 256 when there is more than one segment); workspace for the total width
hipError_t launch_project_mfma_segs(const PackLayout &L, const void *packed, const ColSegs &W,
                                   void *ws, hipStream_t s);
hipError_t launch_project_mfma(const PackLayout &L, const void *packed, void *W, int64_t m,
                               int64_t ldw, void *ws, hipStream_t s);

// Record a message for sn_last_error() on the calling thread; returns st.
int32_t set_error(int32_t st, const char *fmt, ...);
// sn_project_weights' checks of everything but the workspace (SN_OK or the
// status, with the message recorded).
int32_t project_args_check(const void *basis, int64_t d, int64_t k, int32_t dt, const void *W,
                           int64_t m, int64_t ldw);

}  // namespace sn
