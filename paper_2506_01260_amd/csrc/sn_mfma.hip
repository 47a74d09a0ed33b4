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
// U staging in LDS: a producer wave
// ---------------------------------------------------------------------------
// Both codec kernels walk U in chunks of CH fragment steps.  Each packed
// layout stores a chunk as contiguous 1 KiB fragments, so a chunk is copied
// verbatim.  One extra wave per workgroup (the producer) copies chunk c+1
// into one of two LDS buffers with direct-to-LDS loads (each lane's 16 bytes
// land at 16 * lane, i.e. the fragment layout) while the compute waves work
// on chunk c from the other buffer; one workgroup barrier per chunk hands the
// buffers over.  The compute waves therefore issue only their own token-row
// loads and output stores, a fixed number per step, and the compiler keeps
// their pipeline full instead of draining it at every chunk boundary.
//
// Barrier protocol (nchunks chunks, buffers b0/b1):
//   producer: copy chunk 0 -> b0, wait, barrier 0; for c in 0..: copy chunk
//             c+1 -> b((c+1)&1), wait, barrier c+1
//   compute:  barrier 0; for c in 0..: work on b(c&1), barrier c+1
// b((c+1)&1) last held chunk c-1, which every compute wave finished before
// barrier c, so the copy issued after barrier c never overwrites live data.
__device__ __forceinline__ void lds_dma_16(const bf16_t *src, u32x4 *dst) {
  __builtin_amdgcn_global_load_lds(static_cast<const void *>(src),
                                   (__attribute__((address_space(3))) void *)(dst), 16, 0, 0);
}

// Copy `frags` 1 KiB fragments starting at src (global) to dst (LDS); called by
// one whole wave.
__device__ __forceinline__ void produce_chunk(const bf16_t *src, u32x4 *dst, int frags,
                                              int lane) {
  for (int f = 0; f < frags; ++f) lds_dma_16(src + f * 512 + lane * 8, dst + f * 64);
  __builtin_amdgcn_s_waitcnt(0);  // vmcnt(0) and lgkmcnt(0): the copies have landed
}

__device__ __forceinline__ u32x4 lds_frag(const u32x4 *buf, int frag, int lane) {
  return buf[frag * 64 + lane];
}

// ---------------------------------------------------------------------------
// compress
// ---------------------------------------------------------------------------
// Workgroup = W compute waves + 1 producer wave; compute wave w owns NT tiles
// of 16 tokens and contracts the whole of d for them, so no cross-wave
// reduction is needed.  The U fragments of the current d-chunk come from LDS;
// D steps of token rows are in flight per wave (a register ring).
template <int NT, bool HE, bool HP>
struct CData {
  u32x4 x[NT];
  u32x4 e[HE ? NT : 1];
  u32x4 p[HP ? NT : 1];
};

template <int NT, bool HE, bool HP>
__device__ __forceinline__ void c_load(CData<NT, HE, HP> &st, const TokRows<HE, HP> (&rows)[NT],
                                       int s) {
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    st.x[nt] = ld16(rows[nt].x + 32 * s);
    if (HE) st.e[nt] = ld16(rows[nt].e + 32 * s);
    if (HP) st.p[nt] = ld16(rows[nt].p + 32 * s);
  }
}

template <int KT, int NT, bool HE, bool HP>
__device__ __forceinline__ void c_compute(const CData<NT, HE, HP> &st, const u32x4 *ubuf,
                                          int local_step, int lane, f32x4 (&acc)[KT][NT]) {
#pragma unroll
  for (int t = 0; t < KT; ++t) {
    const u32x4 a = lds_frag(ubuf, local_step * KT + t, lane);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      acc[t][nt] = mfma(a, st.x[nt], acc[t][nt]);
      if (HP) acc[t][nt] = mfma(a, neg8(st.p[nt]), acc[t][nt]);
      if (HE) acc[t][nt] = mfma(a, neg8(st.e[nt]), acc[t][nt]);
    }
  }
}

template <int KT>
constexpr int c_chunk_steps() { return KT <= 4 ? 8 : 4; }

template <int KT, int NT, bool HE, bool HP>
constexpr int c_depth() { return (NT * (1 + HE + HP)) <= 1 ? c_chunk_steps<KT>() : 4; }

template <int KT, int NT, int W, bool HE, bool HP>
__global__ __launch_bounds__(64 * (W + 1)) void compress_mfma_kernel(
    const bf16_t *__restrict__ kfrag, int64_t d, int64_t k, const bf16_t *__restrict__ X,
    int64_t N, int64_t ldx, IdArgs ids, bf16_t *__restrict__ C, int64_t ldc, int cvec) {
  constexpr int CH = c_chunk_steps<KT>();
  constexpr int D = c_depth<KT, NT, HE, HP>();
  static_assert(CH % D == 0, "chunk must be a multiple of the depth");
  constexpr int CHUNK_FRAGS = CH * KT;
  __shared__ u32x4 ubuf[2][CHUNK_FRAGS * 64];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int steps = static_cast<int>(d / 32);
  const int nchunks = (steps + CH - 1) / CH;
  // Workgroups start at different d-chunks (wrapping around) so the rows in
  // flight across the chip are not all read at the same column offset.
  const int rot = (steps % CH == 0) ? static_cast<int>(blockIdx.x % nchunks) * CH : 0;
  auto phys = [&](int si) { const int v = si + rot; return v >= steps ? v - steps : v; };

  if (wave == W) {  // producer
    auto copy = [&](int cs) {
      const int c0 = phys(cs * CH) / CH;
      const int left = steps - c0 * CH;
      const int frags = (left < CH ? left : CH) * KT;
      produce_chunk(kfrag + static_cast<int64_t>(c0) * CHUNK_FRAGS * 512, ubuf[cs & 1], frags,
                    lane);
    };
    copy(0);
    __syncthreads();
    for (int cs = 0; cs < nchunks; ++cs) {
      if (cs + 1 < nchunks) copy(cs + 1);
      __syncthreads();
    }
    return;
  }

  const int g = lane >> 4, n = lane & 15;
  const int64_t tok0 = (static_cast<int64_t>(blockIdx.x) * W + wave) * (16 * NT);

  TokRows<HE, HP> rows[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
    rows[nt] = tok_rows<HE, HP>(tok0 + 16 * nt + n, N, X, ldx, ids, 8 * g);

  f32x4 acc[KT][NT];
#pragma unroll
  for (int t = 0; t < KT; ++t)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[t][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Loads past the end re-read the last step (cache hits), so every step
  // issues the same loads.
  auto phys_c = [&](int si) { return phys(si < steps ? si : steps - 1); };
  CData<NT, HE, HP> ring[D];
#pragma unroll
  for (int i = 0; i < D; ++i) c_load(ring[i], rows, phys_c(i));

  // Full chunks run a fully unrolled body with no conditional memory
  // operations (so the compiler can count the loads in flight); a partial
  // last chunk (only when d is not a multiple of 32 * CH, and then without
  // rotation) is peeled off after the loop.
  const int nfull = steps / CH;
  for (int cs = 0; cs < nfull; ++cs) {
    __syncthreads();  // chunk cs is in ubuf[cs & 1]
    const u32x4 *ub = ubuf[cs & 1];
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int si = cs * CH + i;
      c_compute<KT>(ring[i % D], ub, i, lane, acc);
      c_load(ring[i % D], rows, phys_c(si + D));
      // keep the refill here: the scheduler would otherwise sink every refill
      // of the chunk to its end and drain the ring
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  if (nfull < nchunks) {
    __syncthreads();
    const u32x4 *ub = ubuf[nfull & 1];
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int si = nfull * CH + i;
      if (si < steps) c_compute<KT>(ring[i % D], ub, i, lane, acc);
      if (si < steps) c_load(ring[i % D], rows, phys_c(si + D));
    }
  }
  __syncthreads();  // matches the producer's last barrier

#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int64_t i = tok0 + 16 * nt + n;
    if (i >= N) continue;
#pragma unroll
    for (int t = 0; t < KT; ++t) {
      const f32x4 v = acc[t][nt];
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
}

// ---------------------------------------------------------------------------
// decompress
// ---------------------------------------------------------------------------
// Workgroup = W compute waves + 1 producer wave; compute wave w owns NT tiles
// of 16 tokens, keeps their C values (the B operand) in registers and writes
// whole output rows.  The U fragments (A operand) of the current chunk of row
// groups come from LDS; D groups of embedding rows are in flight per wave.
// With embedding terms the output is written with non-temporal stores, so the
// output stream does not push the gathered rows out of the caches.
template <int NT, bool HE, bool HP>
struct DData {
  u32x4 e[HE ? NT : 1];
  u32x4 p[HP ? NT : 1];
};

template <int NT, bool HE, bool HP>
__device__ __forceinline__ void d_load(DData<NT, HE, HP> &st, const TokRows<HE, HP> (&rows)[NT],
                                       int p) {
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    if (HP) st.p[nt] = ld16(rows[nt].p + 32 * p);
    if (HE) st.e[nt] = ld16(rows[nt].e + 32 * p);
  }
}

// Stores are unconditional: a lane past the last token serves a copy of
// token N-1 (same C row, same embedding rows, same instruction sequence), so
// it writes the very bytes the lane that owns token N-1 writes.  Keeping the
// store count fixed lets the compiler count outstanding memory operations.
template <int KS, int NT, bool HE, bool HP, bool NTSTORE>
__device__ __forceinline__ void d_compute_store(const DData<NT, HE, HP> &st, const u32x4 *ubuf,
                                                int local_group, int lane,
                                                const u32x4 (&b)[NT][KS],
                                                bf16_t *const (&xout)[NT], int p) {
  u32x4 a[2][KS];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int q = 0; q < KS; ++q) a[h][q] = lds_frag(ubuf, (local_group * 2 + h) * KS + q, lane);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    f32x4 lo = {0.f, 0.f, 0.f, 0.f}, hi = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < KS; ++q) {
      lo = mfma(a[0][q], b[nt][q], lo);
      hi = mfma(a[1][q], b[nt][q], hi);
    }
    // lane holds X[token, 32 p + 8 g + 0..3] in lo and + 4..7 in hi
    float o[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    if (HP) {
      const uint32_t w[4] = {st.p[nt].x, st.p[nt].y, st.p[nt].z, st.p[nt].w};
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        o[2 * e2] += bf_lo(w[e2]);
        o[2 * e2 + 1] += bf_hi(w[e2]);
      }
    }
    if (HE) {
      const uint32_t w[4] = {st.e[nt].x, st.e[nt].y, st.e[nt].z, st.e[nt].w};
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        o[2 * e2] += bf_lo(w[e2]);
        o[2 * e2 + 1] += bf_hi(w[e2]);
      }
    }
    const u32x4 v = {pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]), pack_bf16x2(o[4], o[5]),
                     pack_bf16x2(o[6], o[7])};
    u32x4 *dst = reinterpret_cast<u32x4 *>(xout[nt] + 32 * p);
    if (NTSTORE)
      __builtin_nontemporal_store(v, dst);
    else
      *dst = v;
  }
}

template <int KS>
constexpr int d_chunk_groups() { return KS <= 2 ? 8 : 4; }

template <int NT, bool HE, bool HP>
constexpr int d_depth() { return (NT * (HE + HP)) <= 2 ? 4 : 2; }

template <int KS, int NT, int W, bool HE, bool HP>
__global__ __launch_bounds__(64 * (W + 1)) void decompress_mfma_kernel(
    const bf16_t *__restrict__ rfrag, int64_t d, int64_t k, const bf16_t *__restrict__ C,
    int64_t N, int64_t ldc, IdArgs ids, bf16_t *__restrict__ X, int64_t ldx, int cvec) {
  constexpr int CH = d_chunk_groups<KS>();
  constexpr int D = d_depth<NT, HE, HP>();
  static_assert(CH % D == 0, "chunk must be a multiple of the depth");
  constexpr int CHUNK_FRAGS = CH * 2 * KS;
  constexpr bool NTSTORE = HE || HP;
  __shared__ u32x4 ubuf[2][CHUNK_FRAGS * 64];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int groups = static_cast<int>(d / 32);
  const int nchunks = (groups + CH - 1) / CH;
  const int rot = (groups % CH == 0) ? static_cast<int>(blockIdx.x % nchunks) * CH : 0;
  auto phys = [&](int si) { const int v = si + rot; return v >= groups ? v - groups : v; };

  if (wave == W) {  // producer
    auto copy = [&](int cs) {
      const int c0 = phys(cs * CH) / CH;
      const int left = groups - c0 * CH;
      const int frags = (left < CH ? left : CH) * 2 * KS;
      produce_chunk(rfrag + static_cast<int64_t>(c0) * CHUNK_FRAGS * 512, ubuf[cs & 1], frags,
                    lane);
    };
    copy(0);
    __syncthreads();
    for (int cs = 0; cs < nchunks; ++cs) {
      if (cs + 1 < nchunks) copy(cs + 1);
      __syncthreads();
    }
    return;
  }

  const int g = lane >> 4, n = lane & 15;
  const int64_t tok0 = (static_cast<int64_t>(blockIdx.x) * W + wave) * (16 * NT);

  // B operand: C[token, 32 q + 8 g + e]
  u32x4 b[NT][KS];
  TokRows<HE, HP> rows[NT];
  bf16_t *xout[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int64_t it = tok0 + 16 * nt + n;
    const int64_t i = it < N ? it : N - 1;  // padding lanes serve a copy of token N-1
    rows[nt] = tok_rows<HE, HP>(it, N, X, ldx, ids, 8 * g);
    xout[nt] = X + i * ldx + 8 * g;
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

  auto phys_c = [&](int si) { return phys(si < groups ? si : groups - 1); };
  DData<NT, HE, HP> ring[D];
#pragma unroll
  for (int i = 0; i < D; ++i) d_load(ring[i], rows, phys_c(i));

  const int nfull = groups / CH;
  for (int cs = 0; cs < nfull; ++cs) {
    __syncthreads();  // chunk cs is in ubuf[cs & 1]
    const u32x4 *ub = ubuf[cs & 1];
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int si = cs * CH + i;
      d_compute_store<KS, NT, HE, HP, NTSTORE>(ring[i % D], ub, i, lane, b, xout, phys(si));
      d_load(ring[i % D], rows, phys_c(si + D));
      __builtin_amdgcn_sched_barrier(0);  // keep the refill here (see compress)
    }
  }
  if (nfull < nchunks) {
    __syncthreads();
    const u32x4 *ub = ubuf[nfull & 1];
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int si = nfull * CH + i;
      if (si < groups) {
        d_compute_store<KS, NT, HE, HP, NTSTORE>(ring[i % D], ub, i, lane, b, xout, phys(si));
        d_load(ring[i % D], rows, phys_c(si + D));
      }
    }
  }
  __syncthreads();  // matches the producer's last barrier
}

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

bool tables_ok(const IdArgs &ids) {
  if (ids.E && (!aligned16(ids.E) || ids.lde % 8 != 0)) return false;
  if (ids.P && (!aligned16(ids.P) || ids.ldp % 8 != 0)) return false;
  return true;
}

// Token-tile geometry: waves per workgroup W and tiles per wave NT, chosen so
// the grid has at least ~2 workgroups per CU.
struct Geometry {
  int w, nt;
};

Geometry pick_geometry(int64_t) {
  // 4 compute waves of one 16-token tile each: 64 tokens per workgroup, so a
  // 32768-token batch fills 256 CUs with 2 workgroups each.
  return {4, 1};
}

template <int KT, int NT, int W, bool HE, bool HP>
void launch_c(const bf16_t *kf, const PackLayout &L, const void *X, int64_t N, int64_t ldx,
              const IdArgs &ids, void *C, int64_t ldc, int cvec, hipStream_t s) {
  dim3 grid(static_cast<unsigned>(ceil_div(N, 16 * NT * W)));
  compress_mfma_kernel<KT, NT, W, HE, HP><<<grid, 64 * (W + 1), 0, s>>>(
      kf, L.d, L.k, static_cast<const bf16_t *>(X), N, ldx, ids, static_cast<bf16_t *>(C), ldc,
      cvec);
}

template <int KT, int NT, int W>
void launch_c_emb(const bf16_t *kf, const PackLayout &L, const void *X, int64_t N, int64_t ldx,
                  const IdArgs &ids, void *C, int64_t ldc, int cvec, hipStream_t s) {
  const bool he = ids.E != nullptr, hp = ids.P != nullptr;
  if (he && hp)
    launch_c<KT, NT, W, true, true>(kf, L, X, N, ldx, ids, C, ldc, cvec, s);
  else if (he)
    launch_c<KT, NT, W, true, false>(kf, L, X, N, ldx, ids, C, ldc, cvec, s);
  else if (hp)
    launch_c<KT, NT, W, false, true>(kf, L, X, N, ldx, ids, C, ldc, cvec, s);
  else
    launch_c<KT, NT, W, false, false>(kf, L, X, N, ldx, ids, C, ldc, cvec, s);
}

template <int KT>
void launch_c_geo(const bf16_t *kf, const PackLayout &L, const void *X, int64_t N, int64_t ldx,
                  const IdArgs &ids, void *C, int64_t ldc, int cvec, hipStream_t s) {
  const Geometry geo = pick_geometry(N);
  if (geo.nt == 2)
    launch_c_emb<KT, 2, 4>(kf, L, X, N, ldx, ids, C, ldc, cvec, s);
  else
    launch_c_emb<KT, 1, 4>(kf, L, X, N, ldx, ids, C, ldc, cvec, s);
}

template <int KS, int NT, int W, bool HE, bool HP>
void launch_d(const bf16_t *rf, const PackLayout &L, const void *C, int64_t N, int64_t ldc,
              const IdArgs &ids, void *X, int64_t ldx, int cvec, hipStream_t s) {
  dim3 grid(static_cast<unsigned>(ceil_div(N, 16 * NT * W)));
  decompress_mfma_kernel<KS, NT, W, HE, HP><<<grid, 64 * (W + 1), 0, s>>>(
      rf, L.d, L.k, static_cast<const bf16_t *>(C), N, ldc, ids, static_cast<bf16_t *>(X), ldx,
      cvec);
}

template <int KS, int NT, int W>
void launch_d_emb(const bf16_t *rf, const PackLayout &L, const void *C, int64_t N, int64_t ldc,
                  const IdArgs &ids, void *X, int64_t ldx, int cvec, hipStream_t s) {
  const bool he = ids.E != nullptr, hp = ids.P != nullptr;
  if (he && hp)
    launch_d<KS, NT, W, true, true>(rf, L, C, N, ldc, ids, X, ldx, cvec, s);
  else if (he)
    launch_d<KS, NT, W, true, false>(rf, L, C, N, ldc, ids, X, ldx, cvec, s);
  else if (hp)
    launch_d<KS, NT, W, false, true>(rf, L, C, N, ldc, ids, X, ldx, cvec, s);
  else
    launch_d<KS, NT, W, false, false>(rf, L, C, N, ldc, ids, X, ldx, cvec, s);
}

template <int KS>
void launch_d_geo(const bf16_t *rf, const PackLayout &L, const void *C, int64_t N, int64_t ldc,
                  const IdArgs &ids, void *X, int64_t ldx, int cvec, hipStream_t s) {
  const Geometry geo = pick_geometry(N);
  if (geo.nt == 2)
    launch_d_emb<KS, 2, 4>(rf, L, C, N, ldc, ids, X, ldx, cvec, s);
  else
    launch_d_emb<KS, 1, 4>(rf, L, C, N, ldc, ids, X, ldx, cvec, s);
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
  switch (L.kt) {
    case 1: launch_c_geo<1>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 2: launch_c_geo<2>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 3: launch_c_geo<3>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 4: launch_c_geo<4>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 5: launch_c_geo<5>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 6: launch_c_geo<6>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 7: launch_c_geo<7>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
    case 8: launch_c_geo<8>(kf, L, X, N, ldx, ids, C, ldc, cvec, s); break;
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
  switch (L.ks) {
    case 1: launch_d_geo<1>(rf, L, C, N, ldc, ids, X, ldx, cvec, s); break;
    case 2: launch_d_geo<2>(rf, L, C, N, ldc, ids, X, ldx, cvec, s); break;
    case 3: launch_d_geo<3>(rf, L, C, N, ldc, ids, X, ldx, cvec, s); break;
    case 4: launch_d_geo<4>(rf, L, C, N, ldc, ids, X, ldx, cvec, s); break;
    default: return hipErrorNotSupported;
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// weight projection W <- U (U^T W), three passes
// ---------------------------------------------------------------------------
//  pass 1  Tp[split][c][j] = sum over the split's rows r of U[r, j] W[r, c]
//          D[j, c] = A[j, r] B[r, c] with A = kfrag.  Lane (g, n) loads the
//          8-byte pieces W[32 s + 8 g + e, cb + 4 n .. +3], e = 0..7 (16 lanes
//          cover 128 contiguous bytes of a row), and transposes that 8 x 4
//          block in registers into four B operands: MFMA instance q serves
//          columns cb + 4 n + q.  The four waves of a workgroup split the rows
//          and are summed through LDS in a fixed order.
//  pass 2  T = sum of the splits (fixed order), split into bf16 hi + lo so the
//          second contraction sees T to ~16 significant bits.
//  pass 3  W[r, c] = sum_j U[r, j] T[j, c]; D[c, r] = A[c, j] B[j, r] with
//          A = T rows (column order chosen so a lane holds 8 consecutive
//          columns of one row: 16-byte stores) and B = rfrag.
// W is read only by pass 1 and written only by pass 3 (stream order), so the
// update is in place.

namespace {

constexpr int kProjCols = 64;  // columns per workgroup in passes 1 and 3

struct ProjPlan {
  int64_t m_pad;      // m rounded up to kProjCols
  int kp;             // 16 * kt: fp32 row length of Tp
  int kp32;           // 32 * ks: bf16 row length of Th / Tl
  int dsplit;         // row splits in pass 1
  int64_t rows_per_split;
  size_t off_tp, off_th, off_tl, total;
};

ProjPlan proj_plan(int64_t d, int kt, int ks, int64_t m) {
  ProjPlan P;
  P.m_pad = ceil_div(m, kProjCols) * kProjCols;
  P.kp = 16 * kt;
  P.kp32 = 32 * ks;
  const int64_t slabs = P.m_pad / kProjCols;
  int64_t ds = ceil_div(256, slabs);           // aim for >= 256 workgroups
  const int64_t max_ds = d / 128;               // >= 32 rows per wave
  if (ds > max_ds) ds = max_ds;
  if (ds > 8) ds = 8;
  if (ds < 1) ds = 1;
  P.rows_per_split = ceil_div(ceil_div(d, ds), 128) * 128;
  P.dsplit = static_cast<int>(ceil_div(d, P.rows_per_split));
  size_t off = 0;
  P.off_tp = off;
  off = align256(off + static_cast<size_t>(P.dsplit) * P.m_pad * P.kp * sizeof(float));
  P.off_th = off;
  off = align256(off + static_cast<size_t>(P.m_pad) * P.kp32 * 2);
  P.off_tl = off;
  off = align256(off + static_cast<size_t>(P.m_pad) * P.kp32 * 2);
  P.total = off;
  return P;
}

template <int KT>
__global__ __launch_bounds__(kBlock) void project_pass1_kernel(
    const bf16_t *__restrict__ kfrag, int64_t d, const bf16_t *__restrict__ W, int64_t m,
    int64_t ldw, int64_t rows_per_split, int64_t m_pad, float *__restrict__ Tp) {
  __shared__ f32x4 red[KT][4][64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int g = lane >> 4, n = lane & 15;
  const int64_t cb = static_cast<int64_t>(blockIdx.x) * kProjCols;
  const int split = blockIdx.y;
  const int64_t col = cb + 4 * n;
  const bool cvalid = col < m;  // m % 8 == 0: all four columns are valid

  const int steps = static_cast<int>(rows_per_split / 32);
  const int sb = static_cast<int>(split * (rows_per_split / 32));
  const int send = static_cast<int>(d / 32);
  int s0 = sb + steps * wave / kWaves;
  int s1 = sb + steps * (wave + 1) / kWaves;
  if (s1 > send) s1 = send;

  f32x4 acc[KT][4];
#pragma unroll
  for (int t = 0; t < KT; ++t)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[t][q] = f32x4{0.f, 0.f, 0.f, 0.f};

  const bf16_t *wcol = W + col;
  const bf16_t *ufrag = kfrag + lane * 8;
  for (int s = s0; s < s1; ++s) {
    u32x2 v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int64_t r = 32 * static_cast<int64_t>(s) + 8 * g + e;
      v[e] = cvalid ? *reinterpret_cast<const u32x2 *>(wcol + r * ldw) : u32x2{0u, 0u};
    }
    u32x4 b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const u32x2 lo = v[2 * i], hi = v[2 * i + 1];
      b[0][i] = (lo.x & 0xFFFFu) | (hi.x << 16);
      b[1][i] = (lo.x >> 16) | (hi.x & 0xFFFF0000u);
      b[2][i] = (lo.y & 0xFFFFu) | (hi.y << 16);
      b[3][i] = (lo.y >> 16) | (hi.y & 0xFFFF0000u);
    }
#pragma unroll
    for (int t = 0; t < KT; ++t) {
      const u32x4 a = ld16(ufrag + (static_cast<int64_t>(s) * KT + t) * 512);
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[t][q] = mfma(a, b[q], acc[t][q]);
    }
  }

  // fixed-order reduction: acc0 + (acc1 + (acc2 + acc3))
  for (int w = kWaves - 1; w >= 1; --w) {
    if (wave == w) {
#pragma unroll
      for (int t = 0; t < KT; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          f32x4 v = acc[t][q];
          if (w < kWaves - 1) v += red[t][q][lane];
          red[t][q][lane] = v;
        }
    }
    __syncthreads();
  }
  if (wave == 0 && cvalid) {
    // lane holds T[16 t + 4 g + i][col + q]
#pragma unroll
    for (int t = 0; t < KT; ++t)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x4 v = acc[t][q] + red[t][q][lane];
        float *dst = Tp + ((static_cast<int64_t>(split) * m_pad + col + q) * (16 * KT)) + 16 * t + 4 * g;
        *reinterpret_cast<f32x4 *>(dst) = v;
      }
  }
}

// pass 2: one thread per (column c, j): sum the splits, split into hi / lo.
__global__ __launch_bounds__(256) void project_pass2_kernel(const float *__restrict__ Tp,
                                                            int dsplit, int64_t m, int64_t m_pad,
                                                            int kp, int kp32,
                                                            bf16_t *__restrict__ Th,
                                                            bf16_t *__restrict__ Tl) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= m_pad * kp32) return;
  const int64_t c = idx / kp32;
  const int j = static_cast<int>(idx - c * kp32);
  float v = 0.0f;
  if (c < m && j < kp) {
    Dot2 acc;
    for (int sp = 0; sp < dsplit; ++sp) acc.add(Tp[(sp * m_pad + c) * kp + j]);
    v = acc.value();
  }
  const bf16_t hi = from_f32<bf16_t>(v);
  const bf16_t lo = from_f32<bf16_t>(v - to_f32(hi));
  Th[idx] = hi;
  Tl[idx] = lo;
}

template <int KS>
__global__ __launch_bounds__(kBlock) void project_pass3_kernel(
    const bf16_t *__restrict__ rfrag, int64_t d, const bf16_t *__restrict__ Th,
    const bf16_t *__restrict__ Tl, bf16_t *__restrict__ W, int64_t m, int64_t ldw,
    int64_t rows_per_block) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int g = lane >> 4, n = lane & 15;
  const int64_t cb = static_cast<int64_t>(blockIdx.x) * kProjCols;

  // A operands: M-tile a covers columns cb + 32 (a / 2) + 8 (mm / 4) + 4 (a % 2) + mm % 4
  u32x4 ah[4][KS], al[4][KS];
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const int64_t crow = cb + 32 * (a >> 1) + 8 * (n >> 2) + 4 * (a & 1) + (n & 3);
#pragma unroll
    for (int q = 0; q < KS; ++q) {
      ah[a][q] = ld16(Th + crow * (32 * KS) + 32 * q + 8 * g);
      al[a][q] = ld16(Tl + crow * (32 * KS) + 32 * q + 8 * g);
    }
  }

  const int64_t r_begin = static_cast<int64_t>(blockIdx.y) * rows_per_block;
  const int gb = static_cast<int>(r_begin / 32);
  const int gcount = static_cast<int>(rows_per_block / 32);
  int p0 = gb + gcount * wave / kWaves;
  int p1 = gb + gcount * (wave + 1) / kWaves;
  const int pend = static_cast<int>(d / 32);
  if (p1 > pend) p1 = pend;
  const bf16_t *ufrag = rfrag + lane * 8;

  for (int p = p0; p < p1; ++p) {
    u32x4 b[2][KS];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int q = 0; q < KS; ++q)
        b[h][q] = ld16(ufrag + ((static_cast<int64_t>(p) * 2 + h) * KS + q) * 512);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t r = 32 * static_cast<int64_t>(p) + 8 * (n >> 2) + 4 * h + (n & 3);
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        f32x4 o[2];
#pragma unroll
        for (int a2 = 0; a2 < 2; ++a2) {
          const int a = 2 * half + a2;
          f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int q = 0; q < KS; ++q) {
            acc = mfma(ah[a][q], b[h][q], acc);
            acc = mfma(al[a][q], b[h][q], acc);
          }
          o[a2] = acc;
        }
        // lane holds W[r, cb + 32 half + 8 g + 0..7]
        const int64_t c0 = cb + 32 * half + 8 * g;
        if (c0 < m) {
          *reinterpret_cast<u32x4 *>(W + r * ldw + c0) =
              u32x4{pack_bf16x2(o[0].x, o[0].y), pack_bf16x2(o[0].z, o[0].w),
                    pack_bf16x2(o[1].x, o[1].y), pack_bf16x2(o[1].z, o[1].w)};
        }
      }
    }
  }
}

template <int KT>
void launch_p1(const ProjPlan &P, const bf16_t *kf, int64_t d, const bf16_t *W, int64_t m,
               int64_t ldw, float *Tp, hipStream_t s) {
  dim3 grid(static_cast<unsigned>(P.m_pad / kProjCols), static_cast<unsigned>(P.dsplit));
  project_pass1_kernel<KT><<<grid, kBlock, 0, s>>>(kf, d, W, m, ldw, P.rows_per_split, P.m_pad,
                                                   Tp);
}

template <int KS>
void launch_p3(const ProjPlan &P, const bf16_t *rf, int64_t d, const bf16_t *Th,
               const bf16_t *Tl, bf16_t *W, int64_t m, int64_t ldw, hipStream_t s) {
  const int64_t slabs = P.m_pad / kProjCols;
  int64_t rsplit = ceil_div(512, slabs);
  const int64_t max_rs = d / 128;
  if (rsplit > max_rs) rsplit = max_rs;
  if (rsplit < 1) rsplit = 1;
  const int64_t rows = ceil_div(ceil_div(d, rsplit), 128) * 128;
  rsplit = ceil_div(d, rows);
  dim3 grid(static_cast<unsigned>(slabs), static_cast<unsigned>(rsplit));
  project_pass3_kernel<KS><<<grid, kBlock, 0, s>>>(rf, d, Th, Tl, W, m, ldw, rows);
}

}  // namespace

size_t project_workspace_mfma(int64_t d, int64_t k, int64_t m) {
  const int kt = static_cast<int>(ceil_div(k, 16)), ks = static_cast<int>(ceil_div(k, 32));
  return proj_plan(d, kt, ks, m).total;
}

bool project_mfma_ok(const PackLayout &L, const void *W, int64_t m, int64_t ldw) {
  return L.mfma && aligned16(W) && ldw % 8 == 0 && m % 8 == 0 && L.d % 128 == 0;
}

hipError_t launch_project_mfma(const PackLayout &L, const void *packed, void *Wv, int64_t m,
                               int64_t ldw, void *ws, hipStream_t s) {
  const ProjPlan P = proj_plan(L.d, L.kt, L.ks, m);
  const char *base = static_cast<const char *>(packed);
  const bf16_t *kf = reinterpret_cast<const bf16_t *>(base + L.off_kfrag);
  const bf16_t *rf = reinterpret_cast<const bf16_t *>(base + L.off_rfrag);
  char *w = static_cast<char *>(ws);
  float *Tp = reinterpret_cast<float *>(w + P.off_tp);
  bf16_t *Th = reinterpret_cast<bf16_t *>(w + P.off_th);
  bf16_t *Tl = reinterpret_cast<bf16_t *>(w + P.off_tl);
  bf16_t *W = static_cast<bf16_t *>(Wv);
  switch (L.kt) {
    case 1: launch_p1<1>(P, kf, L.d, W, m, ldw, Tp, s); break;
    case 2: launch_p1<2>(P, kf, L.d, W, m, ldw, Tp, s); break;
    case 3: launch_p1<3>(P, kf, L.d, W, m, ldw, Tp, s); break;
    case 4: launch_p1<4>(P, kf, L.d, W, m, ldw, Tp, s); break;
    case 5: launch_p1<5>(P, kf, L.d, W, m, ldw, Tp, s); break;
    case 6: launch_p1<6>(P, kf, L.d, W, m, ldw, Tp, s); break;
    case 7: launch_p1<7>(P, kf, L.d, W, m, ldw, Tp, s); break;
    case 8: launch_p1<8>(P, kf, L.d, W, m, ldw, Tp, s); break;
    default: return hipErrorNotSupported;
  }
  const int64_t n2 = P.m_pad * P.kp32;
  project_pass2_kernel<<<dim3(static_cast<unsigned>(ceil_div(n2, 256))), 256, 0, s>>>(
      Tp, P.dsplit, m, P.m_pad, P.kp, P.kp32, Th, Tl);
  switch (L.ks) {
    case 1: launch_p3<1>(P, rf, L.d, Th, Tl, W, m, ldw, s); break;
    case 2: launch_p3<2>(P, rf, L.d, Th, Tl, W, m, ldw, s); break;
    case 3: launch_p3<3>(P, rf, L.d, Th, Tl, W, m, ldw, s); break;
    case 4: launch_p3<4>(P, rf, L.d, Th, Tl, W, m, ldw, s); break;
    default: return hipErrorNotSupported;
  }
  return hipGetLastError();
}

}  // namespace sn
