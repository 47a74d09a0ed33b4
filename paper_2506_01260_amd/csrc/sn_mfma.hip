// bf16 codec kernels on the gfx950 matrix cores (v_mfma_f32_16x16x32_bf16).
//
// MFMA 16x16x32 operand layout (wave64): lane l = 16 g + n (g = l / 16,
// n = l % 16) supplies 8 consecutive K values of row n of A and of column n of
// B, and receives D[4 g + i][n], i = 0..3.  The K values a lane supplies for A
// and for B are the same 8 indices, so any fixed assignment of (g, e) to
// contraction indices gives the same sum; the kernels pick the one under which
// each lane reads 16 contiguous bytes of a token's row.
//
// compress   D[j, token] = sum_r U[r, j] * (X - P[pos] - E[tok])[token, r]
//            A = U fragment (packed "kfrag"), B = 8 contiguous bf16 of a row.
//            The embedding terms enter as extra MFMAs on sign-flipped rows, so
//            X - P - E is never rounded: every bf16 x bf16 product is exact
//            and all sums are fp32.
// decompress D[r, token] = sum_j U[r, j] * C[token, j], then + P[pos] + E[tok]
//            A = U rows (packed "rfrag", row order chosen so a lane's 8 outputs
//            are 8 consecutive d of one token), B = 8 consecutive C values.
#include "sn_device.h"
#include "sn_internal.h"

namespace sn {

namespace {

constexpr int kWaves = 4;  // waves per workgroup
constexpr int kBlock = 64 * kWaves;

__device__ __forceinline__ u32x4 ld16(const bf16_t *p) {
  return *reinterpret_cast<const u32x4 *>(p);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ f32x4 mfma(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

// Negate 8 packed bf16 values (flip their sign bits).
__device__ __forceinline__ u32x4 neg8(u32x4 v) {
  const uint32_t s = 0x80008000u;
  return u32x4{v.x ^ s, v.y ^ s, v.z ^ s, v.w ^ s};
}

// Row pointers of the token a lane serves; tokens past N reuse row N-1 for
// loads (their results are never stored).
template <bool HE, bool HP>
struct TokRows {
  const bf16_t *x;
  const bf16_t *e;
  const bf16_t *p;
};

template <bool HE, bool HP>
__device__ __forceinline__ TokRows<HE, HP> tok_rows(int64_t tok_idx, int64_t N,
                                                    const bf16_t *X, int64_t ldx,
                                                    const IdArgs &a, int col) {
  const int64_t i = tok_idx < N ? tok_idx : N - 1;
  TokRows<HE, HP> r;
  r.x = X + i * ldx + col;
  r.e = nullptr;
  r.p = nullptr;
  if (HE) {
    const int64_t t = clamp_id(a.tok[i], a.vocab, a.err_flag, 1);
    r.e = static_cast<const bf16_t *>(a.E) + t * a.lde + col;
  }
  if (HP) {
    int64_t p = a.pos ? static_cast<int64_t>(a.pos[i]) : i % a.seq_len;
    p = clamp_id(p, a.n_pos, a.err_flag, 2);
    r.p = static_cast<const bf16_t *>(a.P) + p * a.ldp + col;
  }
  return r;
}

// ---------------------------------------------------------------------------
// compress
// ---------------------------------------------------------------------------
// Workgroup = 4 waves on one group of 16*NT tokens; wave w contracts the w-th
// quarter of d, then the four partial results are summed in LDS in wave order
// (fixed order: deterministic).
template <int KT, int NT, bool HE, bool HP>
__global__ __launch_bounds__(kBlock) void compress_mfma_kernel(
    const bf16_t *__restrict__ kfrag, int64_t d, int64_t k, const bf16_t *__restrict__ X,
    int64_t N, int64_t ldx, IdArgs ids, bf16_t *__restrict__ C, int64_t ldc, int cvec) {
  __shared__ f32x4 red[kWaves][KT][NT][64];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int g = lane >> 4, n = lane & 15;
  const int64_t tok0 = static_cast<int64_t>(blockIdx.x) * (16 * NT);

  TokRows<HE, HP> rows[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
    rows[nt] = tok_rows<HE, HP>(tok0 + 16 * nt + n, N, X, ldx, ids, 8 * g);

  f32x4 acc[KT][NT];
#pragma unroll
  for (int t = 0; t < KT; ++t)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[t][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int steps = static_cast<int>(d / 32);
  const int s0 = steps * wave / kWaves;
  const int s1 = steps * (wave + 1) / kWaves;
  const bf16_t *ufrag = kfrag + lane * 8;

#pragma unroll 2
  for (int s = s0; s < s1; ++s) {
    u32x4 bx[NT], be[NT], bp[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      bx[nt] = ld16(rows[nt].x + 32 * s);
      if (HE) be[nt] = neg8(ld16(rows[nt].e + 32 * s));
      if (HP) bp[nt] = neg8(ld16(rows[nt].p + 32 * s));
    }
#pragma unroll
    for (int t = 0; t < KT; ++t) {
      const u32x4 a = ld16(ufrag + (s * KT + t) * 512);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        acc[t][nt] = mfma(a, bx[nt], acc[t][nt]);
        if (HP) acc[t][nt] = mfma(a, bp[nt], acc[t][nt]);
        if (HE) acc[t][nt] = mfma(a, be[nt], acc[t][nt]);
      }
    }
  }

#pragma unroll
  for (int t = 0; t < KT; ++t)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) red[wave][t][nt][lane] = acc[t][nt];
  __syncthreads();

  // wave w finalises tiles (t, nt) with (t * NT + nt) % 4 == w
  for (int tile = wave; tile < KT * NT; tile += kWaves) {
    const int t = tile / NT, nt = tile % NT;
    f32x4 v = red[0][t][nt][lane];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) v += red[w][t][nt][lane];
    const int64_t i = tok0 + 16 * nt + n;
    if (i >= N) continue;
    const int64_t j = 16 * t + 4 * g;  // this lane holds C[i, j .. j+3]
    bf16_t *dst = C + i * ldc + j;
    if (cvec && j + 4 <= k) {
      *reinterpret_cast<u32x2 *>(dst) = u32x2{pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w)};
    } else {
      const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (j + e < k) dst[e] = from_f32<bf16_t>(vv[e]);
    }
  }
}

// ---------------------------------------------------------------------------
// decompress
// ---------------------------------------------------------------------------
// Workgroup = 4 waves on one group of 16*NT tokens; wave w writes the w-th
// quarter of d.  Each lane keeps its tokens' C values (the B operand) in
// registers for the whole sweep over d.
template <int KS, int NT, bool HE, bool HP>
__global__ __launch_bounds__(kBlock) void decompress_mfma_kernel(
    const bf16_t *__restrict__ rfrag, int64_t d, int64_t k, const bf16_t *__restrict__ C,
    int64_t N, int64_t ldc, IdArgs ids, bf16_t *__restrict__ X, int64_t ldx, int cvec) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int g = lane >> 4, n = lane & 15;
  const int64_t tok0 = static_cast<int64_t>(blockIdx.x) * (16 * NT);

  // B operand: C[token, 32 q + 8 g + e]
  u32x4 b[NT][KS];
  TokRows<HE, HP> rows[NT];
  bool valid[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int64_t it = tok0 + 16 * nt + n;
    valid[nt] = it < N;
    const int64_t i = valid[nt] ? it : N - 1;
    rows[nt] = tok_rows<HE, HP>(it, N, X, ldx, ids, 8 * g);
    rows[nt].x = X + i * ldx + 8 * g;
    const bf16_t *cr = C + i * ldc;
#pragma unroll
    for (int q = 0; q < KS; ++q) {
      const int64_t j = 32 * q + 8 * g;
      if (cvec && j + 8 <= k) {
        b[nt][q] = ld16(cr + j);
      } else {
        uint32_t w[4];
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
          const uint32_t lo = j + 2 * e2 < k ? cr[j + 2 * e2] : 0u;
          const uint32_t hi = j + 2 * e2 + 1 < k ? cr[j + 2 * e2 + 1] : 0u;
          w[e2] = lo | (hi << 16);
        }
        b[nt][q] = u32x4{w[0], w[1], w[2], w[3]};
      }
    }
  }

  const int groups = static_cast<int>(d / 32);
  const int p0 = groups * wave / kWaves;
  const int p1 = groups * (wave + 1) / kWaves;
  const bf16_t *ufrag = rfrag + lane * 8;

#pragma unroll 2
  for (int p = p0; p < p1; ++p) {
    u32x4 a[2][KS];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int q = 0; q < KS; ++q) a[h][q] = ld16(ufrag + ((p * 2 + h) * KS + q) * 512);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      u32x4 ev, pv;
      if (HP) pv = ld16(rows[nt].p + 32 * p);
      if (HE) ev = ld16(rows[nt].e + 32 * p);
      f32x4 lo = {0.f, 0.f, 0.f, 0.f}, hi = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int q = 0; q < KS; ++q) {
        lo = mfma(a[0][q], b[nt][q], lo);
        hi = mfma(a[1][q], b[nt][q], hi);
      }
      // lane holds X[token, 32 p + 8 g + 0..3] in lo and + 4..7 in hi
      float o[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      if (HP) {
        const uint32_t w[4] = {pv.x, pv.y, pv.z, pv.w};
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
          o[2 * e2] += bf_lo(w[e2]);
          o[2 * e2 + 1] += bf_hi(w[e2]);
        }
      }
      if (HE) {
        const uint32_t w[4] = {ev.x, ev.y, ev.z, ev.w};
#pragma unroll
        for (int e2 = 0; e2 < 4; ++e2) {
          o[2 * e2] += bf_lo(w[e2]);
          o[2 * e2 + 1] += bf_hi(w[e2]);
        }
      }
      if (valid[nt]) {
        *reinterpret_cast<u32x4 *>(const_cast<bf16_t *>(rows[nt].x) + 32 * p) =
            u32x4{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]), pack_bf16x2(o[4], o[5]),
                  pack_bf16x2(o[6], o[7])};
      }
    }
  }
}

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

bool tables_ok(const IdArgs &ids) {
  if (ids.E && (!aligned16(ids.E) || ids.lde % 8 != 0)) return false;
  if (ids.P && (!aligned16(ids.P) || ids.ldp % 8 != 0)) return false;
  return true;
}

template <int KT, int NT, bool HE, bool HP>
void launch_c(const bf16_t *kf, const PackLayout &L, const void *X, int64_t N, int64_t ldx,
              const IdArgs &ids, void *C, int64_t ldc, int cvec, hipStream_t s) {
  dim3 grid(static_cast<unsigned>(ceil_div(N, 16 * NT)));
  compress_mfma_kernel<KT, NT, HE, HP><<<grid, kBlock, 0, s>>>(
      kf, L.d, L.k, static_cast<const bf16_t *>(X), N, ldx, ids, static_cast<bf16_t *>(C), ldc,
      cvec);
}

template <int KT, int NT>
void launch_c_emb(const bf16_t *kf, const PackLayout &L, const void *X, int64_t N, int64_t ldx,
                  const IdArgs &ids, void *C, int64_t ldc, int cvec, hipStream_t s) {
  const bool he = ids.E != nullptr, hp = ids.P != nullptr;
  if (he && hp)
    launch_c<KT, NT, true, true>(kf, L, X, N, ldx, ids, C, ldc, cvec, s);
  else if (he)
    launch_c<KT, NT, true, false>(kf, L, X, N, ldx, ids, C, ldc, cvec, s);
  else if (hp)
    launch_c<KT, NT, false, true>(kf, L, X, N, ldx, ids, C, ldc, cvec, s);
  else
    launch_c<KT, NT, false, false>(kf, L, X, N, ldx, ids, C, ldc, cvec, s);
}

template <int KS, int NT, bool HE, bool HP>
void launch_d(const bf16_t *rf, const PackLayout &L, const void *C, int64_t N, int64_t ldc,
              const IdArgs &ids, void *X, int64_t ldx, int cvec, hipStream_t s) {
  dim3 grid(static_cast<unsigned>(ceil_div(N, 16 * NT)));
  decompress_mfma_kernel<KS, NT, HE, HP><<<grid, kBlock, 0, s>>>(
      rf, L.d, L.k, static_cast<const bf16_t *>(C), N, ldc, ids, static_cast<bf16_t *>(X), ldx,
      cvec);
}

template <int KS, int NT>
void launch_d_emb(const bf16_t *rf, const PackLayout &L, const void *C, int64_t N, int64_t ldc,
                  const IdArgs &ids, void *X, int64_t ldx, int cvec, hipStream_t s) {
  const bool he = ids.E != nullptr, hp = ids.P != nullptr;
  if (he && hp)
    launch_d<KS, NT, true, true>(rf, L, C, N, ldc, ids, X, ldx, cvec, s);
  else if (he)
    launch_d<KS, NT, true, false>(rf, L, C, N, ldc, ids, X, ldx, cvec, s);
  else if (hp)
    launch_d<KS, NT, false, true>(rf, L, C, N, ldc, ids, X, ldx, cvec, s);
  else
    launch_d<KS, NT, false, false>(rf, L, C, N, ldc, ids, X, ldx, cvec, s);
}

}  // namespace

bool compress_mfma_ok(const PackLayout &L, const void *X, int64_t ldx, const IdArgs &ids) {
  return L.mfma && aligned16(X) && ldx % 8 == 0 && tables_ok(ids);
}

hipError_t launch_compress_mfma(const PackLayout &L, const void *packed, const void *X,
                                int64_t N, int64_t ldx, const IdArgs &ids, void *C, int64_t ldc,
                                hipStream_t s) {
  const bf16_t *kf =
      reinterpret_cast<const bf16_t *>(static_cast<const char *>(packed) + L.off_kfrag);
  const int cvec = ((reinterpret_cast<uintptr_t>(C) & 7) == 0) && (ldc % 4 == 0);
  constexpr int NT = 2;
  switch (L.kt) {
    case 1: launch_c_emb<1, NT>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 2: launch_c_emb<2, NT>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 3: launch_c_emb<3, NT>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 4: launch_c_emb<4, NT>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 5: launch_c_emb<5, NT>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 6: launch_c_emb<6, NT>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 7: launch_c_emb<7, NT>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 8: launch_c_emb<8, NT>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    default: return hipErrorNotSupported;
  }
  return hipGetLastError();
}

bool decompress_mfma_ok(const PackLayout &L, void *X, int64_t ldx, const IdArgs &ids) {
  return L.mfma && aligned16(X) && ldx % 8 == 0 && tables_ok(ids);
}

hipError_t launch_decompress_mfma(const PackLayout &L, const void *packed, const void *C,
                                  int64_t N, int64_t ldc, const IdArgs &ids, void *X,
                                  int64_t ldx, hipStream_t s) {
  const bf16_t *rf =
      reinterpret_cast<const bf16_t *>(static_cast<const char *>(packed) + L.off_rfrag);
  const int cvec = aligned16(C) && (ldc % 8 == 0);
  constexpr int NT = 2;
  switch (L.ks) {
    case 1: launch_d_emb<1, NT>(rf, L, C, N, ldc, ids, X, ldx, cvec, s); break;
    case 2: launch_d_emb<2, NT>(rf, L, C, N, ldc, ids, X, ldx, cvec, s); break;
    case 3: launch_d_emb<3, NT>(rf, L, C, N, ldc, ids, X, ldx, cvec, s); break;
    case 4: launch_d_emb<4, NT>(rf, L, C, N, ldc, ids, X, ldx, cvec, s); break;
    default: return hipErrorNotSupported;
  }
  return hipGetLastError();
}

// The projection's MFMA path is not built yet: the generic kernels serve it.
size_t project_workspace_mfma(int64_t, int64_t, int64_t) { return 0; }
bool project_mfma_ok(const PackLayout &, const void *, int64_t, int64_t) { return false; }
hipError_t launch_project_mfma(const PackLayout &, const void *, void *, int64_t, int64_t, void *,
                               hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace sn
