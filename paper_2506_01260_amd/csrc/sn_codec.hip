// The bf16 compress kernels on the gfx950 matrix cores (decompress is in
// sn_decompress.hip, the weight projection in sn_project.hip).
//
// compress   C[i, :] = (X[i, :] - P[pos_i, :] - E[tok_i, :]) U      (Sec. 4.3.1, Eq. "subtract")
//            D[j, token] = sum_r U[r, j] * (X - P - E)[token, r], computed as
//            X U + (-P) U + (-E) U in one set of fp32 accumulators (sign-flipped
//            bf16 operands), so X - P - E is never rounded: every bf16 product
//            is exact and every sum is fp32.
// Without tables this is the gradient compress of Sec. 4.4.
//
// compress_kernel (one workgroup = NW compute waves + 3 producer waves, 16 NW
// tokens; NW = 8 where three stage buffers of that width fit in LDS and the
// launch has a workgroup for every CU, else 4):
//
// * Three producer waves copy, for each stage of 64 columns of d, everything
//   the compute waves need into one of NB LDS buffers with direct-to-LDS
//   loads: wave A the tokens' X rows, wave B their T_fixed and P rows,
//   wave C the U fragments of the stage.  Each copy instruction reads 8 rows
//   x 128 contiguous bytes (contiguous row pieces are much cheaper for the
//   memory pipeline than the 16-rows-x-64-bytes pattern of an MFMA operand),
//   and the 16-byte pieces of row r are stored in the order p ^ (r & 7) so
//   that the compute waves' operand reads (16 rows, same piece) spread over
//   the banks.
// * T_fixed rows are copied once per distinct id of the workgroup's tokens
//   (Zipf-distributed ids repeat: about 80 distinct ids per 128 tokens at
//   vocab 32000); the T_fixed producer finds the distinct ids at the start
//   and hands each compute lane the slot of its token's row.
// * Compute wave w owns 16 tokens and the whole of d; it reads operands only
//   from LDS (no global loads in its main loop), so nothing stalls it but the
//   hand-over barrier.
// * NB-deep buffering (as many stage buffers as LDS holds, at most 6): the
//   copies keep NB - 1 stages in flight, which is what sets the kernel's
//   speed (one workgroup per CU); three producers keep each wave's
//   outstanding copies within the 6-bit vmcnt range.  One barrier per stage
//   hands a buffer over.  Workgroups start at different stages (rotation) so
//   the rows in flight across the chip are not read at the same column
//   offsets.  The U fragments of a stage are copied once per workgroup, so
//   eight compute waves (128 tokens) halve their share of the copies.
// * Position-major tiles (positions i mod seq_len, batch a multiple of 4): a
//   16-token tile holds 16/BP consecutive positions of BP batches, so the
//   tile needs only 16/BP positional rows.
//
// stream_compress_kernel (X U with no gathered rows) is described at its
// definition.
#include <atomic>

#include "sn_mfma_common.h"

namespace sn {

namespace {

constexpr int kW = 4;                  // compute waves per workgroup (streaming kernel)
constexpr int kThreads = 64 * (kW + 1);
constexpr int kStageCols = 64;         // d-elements per stage
constexpr int kPieces = 8;             // 16-byte pieces per row per stage
constexpr int kRowsPerCopy = 64 / kPieces;  // rows per direct-to-LDS copy instruction
constexpr int kProd = 3;               // producer waves of compress_kernel
constexpr int kMaxStages = 6;

// threads of a compress_kernel workgroup with NW compute waves
template <int NW>
constexpr int threads_c() { return 64 * (NW + kProd); }
constexpr int kLdsBytes = 160 * 1024;

// 16-byte LDS slot of piece p of row r in a row tile.
__device__ __forceinline__ int slot(int r, int p) { return r * kPieces + (p ^ (r & 7)); }

// Token placement of a launch.
struct Tiling {
  int64_t N;
  int64_t seq;      // positions per sequence (position-major tiles only)
  int bp;           // batches per tile: 1 = token-major, else 4 or 8
  int p_stream;     // copy the P rows non-temporally (beside T_fixed, a large P)
};

// Token of lane n of 16-token tile T (T already clamped to a valid tile);
// token-major tiles past N repeat token N-1.  Position-major tiles cover
// whole sequences, so when the last sequence is short they name tokens at or
// past N: those rows are loaded as token N-1 (load_token) and never stored.
__device__ __forceinline__ int64_t tile_token(const Tiling &tm, int64_t T, int n) {
  if (tm.bp == 1) {
    const int64_t t = 16 * T + n;
    return t < tm.N ? t : tm.N - 1;
  }
  const int pg = 16 / tm.bp;
  const int64_t tpb = tm.seq / pg;
  const int64_t bg = T / tpb, pt = T - bg * tpb;
  return (bg * tm.bp + n % tm.bp) * tm.seq + pt * pg + n / tm.bp;
}

// The token whose rows lane n of tile T loads (always below N).
__device__ __forceinline__ int64_t load_token(const Tiling &tm, int64_t T, int n) {
  const int64_t t = tile_token(tm, T, n);
  return t < tm.N ? t : tm.N - 1;
}

// Tiles of a launch: token-major ceil(N / 16); position-major whole
// sequences, ceil(N / seq) of them (bp x 16 / bp = 16 tokens per tile).
__host__ __device__ __forceinline__ int64_t tile_count(const Tiling &tm) {
  if (tm.bp == 1) return (tm.N + 15) / 16;
  return (tm.N + tm.seq - 1) / tm.seq * (tm.seq / 16);
}

// First position of position-major tile T.
__device__ __forceinline__ int64_t tile_pos0(const Tiling &tm, int64_t T) {
  const int pg = 16 / tm.bp;
  const int64_t tpb = tm.seq / pg;
  return (T % tpb) * pg;
}

// positional rows staged per workgroup: 16/BP per tile in position-major
// order (BP batches per tile), one per token in token-major order (BP = 1)
template <int NW, int BP>
constexpr int p_rows() { return BP > 1 ? NW * (16 / BP) : 16 * NW; }

// ---------------------------------------------------------------------------
// Stage buffer geometry (in 16-byte units) of compress_kernel.
// ---------------------------------------------------------------------------
template <int KT, bool HE, bool HP, int BP, int NW>
struct CGeo {
  static constexpr int tokens = 16 * NW;
  static constexpr int x_off = 0;
  static constexpr int e_off = x_off + tokens * kPieces;
  static constexpr int p_off = e_off + (HE ? tokens * kPieces : 0);
  static constexpr int u_off = p_off + (HP ? p_rows<NW, BP>() * kPieces : 0);
  static constexpr int u_frags = (kStageCols / 32) * KT;
  static constexpr int buf_units = u_off + u_frags * 64;
  // with both tables, the positional rows go with the U fragments so the
  // three producers issue about as many copies each
  static constexpr bool p_with_u = HE && HP;
  // copy instructions per stage of each producer: X; gathered rows; U
  static constexpr int dma_a = tokens / kRowsPerCopy;
  static constexpr int dma_p = HP ? (p_rows<NW, BP>() + kRowsPerCopy - 1) / kRowsPerCopy : 0;
  static constexpr int dma_b = (HE ? tokens / kRowsPerCopy : 0) + (p_with_u ? 0 : dma_p);
  static constexpr int dma_c = u_frags + (p_with_u ? dma_p : 0);
  static constexpr int dmax = dma_a > dma_b ? (dma_a > dma_c ? dma_a : dma_c)
                                            : (dma_b > dma_c ? dma_b : dma_c);
  // as many stages as LDS holds (at most kMaxStages), with (nb - 2) stages of
  // every producer's copies countable by vmcnt
  static constexpr int nb_lds = kLdsBytes / (buf_units * 16);
  static constexpr int nb_cap = nb_lds < kMaxStages ? nb_lds : kMaxStages;
  static constexpr int nb = nb_cap - 2 > 63 / dmax ? 2 + 63 / dmax : nb_cap;
  static_assert(nb >= 3, "at least two stages in flight");
};

// Compute waves per workgroup: 8 while three stage buffers of that width fit
// in LDS (four at k <= 48 with both tables, three above), else 4.
template <int KT, bool HE, bool HP, int BP>
constexpr int nw_of() {
  constexpr int rows = 128 * (HE ? 2 : 1) + (HP ? p_rows<8, BP>() : 0);  // X, T_fixed, P rows
  constexpr int units = rows * kPieces + (kStageCols / 32) * KT * 64;
  return kLdsBytes / (units * 16) >= 3 ? 8 : 4;
}

// ---------------------------------------------------------------------------
// Producer waves
// ---------------------------------------------------------------------------
// Row pointers of the rows this lane copies: row r = 8 i + q of a tile of R
// rows (q = lane / 8); lane (q, m) copies piece m ^ (r & 7) of row r.
template <int R>
struct RowSet {
  const bf16_t *ptr[R / kRowsPerCopy];
};

// STREAM: non-temporal copy (cache-policy bit 1), for rows read exactly once
// (X): it keeps them from evicting the gathered rows, which are reused.
template <int R, bool STREAM = false>
__device__ __forceinline__ void dma_rows(const RowSet<R> &rs, int64_t col, u32x4 *dst, int q,
                                         int m) {
#pragma unroll
  for (int i = 0; i < R / kRowsPerCopy; ++i) {
    const int r = kRowsPerCopy * i + q;
    __builtin_amdgcn_global_load_lds(
        static_cast<const void *>(rs.ptr[i] + col + 8 * (m ^ (r & 7))),
        (__attribute__((address_space(3))) void *)(dst + i * 64), 16, 0, STREAM ? 2 : 0);
  }
}

// dma_rows with the cache policy chosen at run time (a wave-uniform branch
// between two copies whose policy operands differ, which the compiler
// cannot fold into one).
template <int R>
__device__ __forceinline__ void dma_rows_rt(const RowSet<R> &rs, bool stream, int64_t col,
                                            u32x4 *dst, int q, int m) {
  if (stream)
    dma_rows<R, true>(rs, col, dst, q, m);
  else
    dma_rows<R, false>(rs, col, dst, q, m);
}

// The first n (wave-uniform) copies of dma_rows.
template <int R>
__device__ __forceinline__ void dma_rows_n(const RowSet<R> &rs, int n, int64_t col, u32x4 *dst,
                                           int q, int m) {
#pragma unroll
  for (int i = 0; i < R / kRowsPerCopy; ++i) {
    if (i < n) {
      const int r = kRowsPerCopy * i + q;
      __builtin_amdgcn_global_load_lds(
          static_cast<const void *>(rs.ptr[i] + col + 8 * (m ^ (r & 7))),
          (__attribute__((address_space(3))) void *)(dst + i * 64), 16, 0, 0);
    }
  }
}

__device__ __forceinline__ void dma_frags(const bf16_t *src, int frags, u32x4 *dst, int lane) {
  for (int f = 0; f < frags; ++f) lds_dma_16(src + f * 512 + lane * 8, dst + f * 64);
}

// Pointer to the start of row `row` of a table.
__device__ __forceinline__ const bf16_t *row_ptr(const void *base, int64_t ld, int64_t row) {
  return static_cast<const bf16_t *>(base) + row * ld;
}

// Wait until at most `later` stages of PER copies each are outstanding
// (later <= L, a compile-time bound: vmcnt takes an immediate).
template <int PER, int L>
__device__ __forceinline__ void wait_stages(int later) {
  if constexpr (L > 0) {
    if (later >= L) {
      wait_vmcnt<L * PER>();
      return;
    }
    wait_stages<PER, L - 1>(later);
  } else {
    wait_vmcnt<0>();
  }
}

// Wait until at most v (wave-uniform, 0 <= v <= V) copies are outstanding.
template <int V>
__device__ __forceinline__ void wait_vm_upto(int v) {
  if constexpr (V > 0) {
    if (v >= V) {
      wait_vmcnt<V>();
      return;
    }
    wait_vm_upto<V - 1>(v);
  } else {
    wait_vmcnt<0>();
  }
}

// ---------------------------------------------------------------------------
// compress
// ---------------------------------------------------------------------------
// Epilogues: bf16 coefficients; coefficients against projected tables
// (C = X U - (P U)[pos] - (T_fixed U)[tok], the subtraction done on the k
// coefficients of each token); fp32 rows of a projected table (padded to
// 16 ceil(k/16) columns, zero past k).
// The subspace-update epilogue (kEpiGrass) sums each row's off-subspace loss
// term per workgroup and writes the coefficients split into bf16 hi + lo in
// the token contraction's operand layout, plus the bf16 coefficients when an
// output is given (see GrassOut).
enum Epi { kEpiBf16 = 0, kEpiProjected = 1, kEpiF32 = 2, kEpiGrass = 3 };

template <int KT, bool HE, bool HP, int BP, int NW, int EPI>
__global__ __launch_bounds__(threads_c<NW>()) void compress_kernel(const bf16_t *__restrict__ kfrag,
                                                             int64_t d, int64_t k,
                                                             const bf16_t *__restrict__ X,
                                                             int64_t ldx, Tiling tm, IdArgs ids,
                                                             ProjArgs pa, void *__restrict__ Cout,
                                                             int64_t ldc, int cvec, GrassOut go) {
  static_assert(EPI == kEpiBf16 || (!HE && !HP && BP == 1), "projected epilogues have no tables");
  constexpr bool PM = BP > 1;
  constexpr int kTokens = 16 * NW;
  using G = CGeo<KT, HE, HP, BP, NW>;
  constexpr int NB = G::nb;
  __shared__ u32x4 lds[NB * G::buf_units];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int nst = static_cast<int>(d / kStageCols);
  const int rot = static_cast<int>(blockIdx.x % static_cast<unsigned>(nst));
  auto phys = [&](int si) { const int v = si + rot; return v >= nst ? v - nst : v; };
  const int64_t ntiles = tile_count(tm);
  const int64_t T0 = static_cast<int64_t>(blockIdx.x) * NW;

  if (wave >= NW) {  // ------------------------------------------------ producers
    // 0: X rows; 1: T_fixed rows (and P rows with no T_fixed); 2: U fragments
    // (and P rows with both tables)
    const int role = wave - NW;
    const int prole = G::p_with_u ? 2 : 1;  // the producer that copies P rows
    const int q = lane / kPieces, m = lane % kPieces;
    RowSet<kTokens> rx, re;
    RowSet<G::dma_p * kRowsPerCopy> rp;
    // token row r = 16 w + n of the workgroup (tiles past the end repeat the
    // last; rows past N load token N - 1)
    auto token_of = [&](int r) {
      int64_t T = T0 + r / 16;
      T = T < ntiles ? T : ntiles - 1;
      return load_token(tm, T, r % 16);
    };
    if (role == 0) {
#pragma unroll
      for (int i = 0; i < kTokens / kRowsPerCopy; ++i)
        rx.ptr[i] = X + token_of(kRowsPerCopy * i + q) * ldx;
    }
    // T_fixed copies per stage: one per 8 distinct ids
    int ce = G::dma_b;
    if (role == 1 && HE) {
      static_assert(kTokens == 128 || kTokens == 64, "one or two tokens per lane");
      constexpr int TPL = kTokens / 64;  // tokens per lane
      // scratch in the last stage buffer, which no copy touches before the
      // first stage hand-over: ids, slot of each first occurrence, distinct
      // ids in slot order, and each token's slot (read by the compute waves)
      int *scr = reinterpret_cast<int *>(lds + (NB - 1) * G::buf_units + G::e_off);
      int *sid = scr, *sfirst = scr + kTokens, *surow = scr + 2 * kTokens;
      int *smap = scr + 3 * kTokens;
      int id[TPL], f[TPL];
#pragma unroll
      for (int h = 0; h < TPL; ++h) {
        const int64_t t = token_of(lane + 64 * h);
        id[h] = static_cast<int>(clamp_id(ids.tok[t], ids.vocab, ids.err_flag, 1));
        sid[lane + 64 * h] = id[h];
        f[h] = lane + 64 * h;
      }
      // first occurrence of each token's id (same wave: the writes above are
      // visible to these reads)
      for (int j = 0; j < kTokens; j += 4) {
        const int4 v = *reinterpret_cast<const int4 *>(sid + j);
#pragma unroll
        for (int h = 0; h < TPL; ++h) {
          // scanning upwards, the first match is the smallest index
          if (v.w == id[h] && j + 3 < f[h]) f[h] = j + 3;
          if (v.z == id[h] && j + 2 < f[h]) f[h] = j + 2;
          if (v.y == id[h] && j + 1 < f[h]) f[h] = j + 1;
          if (v.x == id[h] && j < f[h]) f[h] = j;
        }
      }
      // slots in token order of the first occurrences
      const uint64_t below = (1ull << lane) - 1ull;
      int u = 0;
#pragma unroll
      for (int h = 0; h < TPL; ++h) {
        const bool first = f[h] == lane + 64 * h;
        const uint64_t mk = __ballot(first);
        const int sl = u + __popcll(mk & below);
        if (first) {
          sfirst[lane + 64 * h] = sl;
          surow[sl] = id[h];
        }
        u += __popcll(mk);
      }
#pragma unroll
      for (int h = 0; h < TPL; ++h) smap[lane + 64 * h] = sfirst[f[h]];
      u = __builtin_amdgcn_readfirstlane(u);
      ce = (u + kRowsPerCopy - 1) / kRowsPerCopy;
#pragma unroll
      for (int i = 0; i < kTokens / kRowsPerCopy; ++i) {
        int r = kRowsPerCopy * i + q;
        r = r < u ? r : u - 1;  // lanes of a part-filled last copy repeat the last row
        re.ptr[i] = row_ptr(ids.E, ids.lde, surow[r]);
      }
    }
    if (role == prole && HP) {
      if (!PM) {
#pragma unroll
        for (int i = 0; i < kTokens / kRowsPerCopy; ++i) {
          const int64_t t = token_of(kRowsPerCopy * i + q);
          int64_t ps = ids.pos ? static_cast<int64_t>(ids.pos[t]) : t % ids.seq_len;
          ps = clamp_id(ps, ids.n_pos, ids.err_flag, 2);
          rp.ptr[i] = row_ptr(ids.P, ids.ldp, ps);
        }
      } else {
        // positional row r = w * pg + rho of the workgroup (rows past NW pg
        // repeat the last one so the copy count stays fixed)
        constexpr int pg = 16 / BP;
#pragma unroll
        for (int i = 0; i < G::dma_p; ++i) {
          int r = kRowsPerCopy * i + q;
          r = r < NW * pg ? r : NW * pg - 1;
          int64_t T = T0 + r / pg;
          T = T < ntiles ? T : ntiles - 1;
          rp.ptr[i] = row_ptr(ids.P, ids.ldp, tile_pos0(tm, T) + r % pg);
        }
      }
    }
    auto issue = [&](int si) {
      u32x4 *b = lds + (si % NB) * G::buf_units;
      const int st = phys(si);
      const int64_t col = static_cast<int64_t>(st) * kStageCols;
      if (role == 0) {
        // non-temporal unless the rows are read again (the subspace update's
        // second pass reads G in reverse order, from the Infinity Cache)
        dma_rows<kTokens, EPI != kEpiGrass>(rx, col, b + G::x_off, q, m);
      } else if (role == 1) {
        if (HE) dma_rows_n(re, ce, col, b + G::e_off, q, m);
        if (HP && !G::p_with_u) dma_rows_rt(rp, tm.p_stream != 0, col, b + G::p_off, q, m);
      } else {
        dma_frags(kfrag + static_cast<int64_t>(st) * G::u_frags * 512, G::u_frags, b + G::u_off,
                  lane);
        if (HP && G::p_with_u) dma_rows_rt(rp, tm.p_stream != 0, col, b + G::p_off, q, m);
      }
    };
    for (int s = 0; s < NB - 1; ++s)
      if (s < nst) issue(s);
    if (HE) lds_barrier();  // the token slots are in LDS
    for (int s = 0; s < nst; ++s) {
      // stage s has landed once at most the later stages in flight are pending
      int later = nst - 1 - s;
      later = later < NB - 2 ? later : NB - 2;
      if (role == 0)
        wait_stages<G::dma_a, NB - 2>(later);
      else if (role == 1 && HE)
        wait_vm_upto<G::dma_b * (NB - 2)>(later * ce);
      else if (role == 1)
        wait_stages<G::dma_b, NB - 2>(later);
      else
        wait_stages<G::dma_c, NB - 2>(later);
      lds_barrier();
      if (s + NB - 1 < nst) issue(s + NB - 1);
    }
    if constexpr (HP && PM) {  // the compute waves' exchange of the positional products
      lds_barrier();
      lds_barrier();
    }
    if constexpr (EPI == kEpiGrass) {  // the compute waves' epilogue exchange
      lds_barrier();
      lds_barrier();
      lds_barrier();
    }
    return;
  }

  // ------------------------------------------------------------ compute waves
  const int g = lane >> 4, n = lane & 15;
  const int xrow = 16 * wave + n;
  const int prow = PM ? wave * (16 / BP) + n / BP : xrow;
  int erow = xrow;  // slot of the token's T_fixed row
  if constexpr (HE) {
    lds_barrier();
    erow = reinterpret_cast<const int *>(lds + (NB - 1) * G::buf_units + G::e_off)[3 * kTokens + xrow];
  }

  f32x4 acc[KT];
#pragma unroll
  for (int t = 0; t < KT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  double sq = 0.0;  // kEpiGrass: sum of squares of the lane's elements of its row

  // Position-major tiles: the workgroup has only PR positional rows, so their
  // products (-P) U are formed once per row rather than once per token: the
  // jobs (P tile pt of 16 rows, column tile t) are dealt to the compute waves
  // (at most two each), and after the last stage every token adds its row's
  // product through LDS.
  constexpr bool kPT = HP && PM;
  constexpr int PR = p_rows<NW, BP>();
  constexpr int NJOB = ((PR + 15) / 16) * KT;
  constexpr int JPW = (NJOB + NW - 1) / NW;
  static_assert(!kPT || JPW <= 2, "at most two positional jobs per wave");
  f32x4 pacc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};

  for (int s = 0; s < nst; ++s) {
    lds_barrier();  // stage s is in buffer s % NB
    const u32x4 *b = lds + (s % NB) * G::buf_units;
#pragma unroll
    for (int j = 0; j < kStageCols / 32; ++j) {
      const int pc = 4 * j + g;
      const u32x4 bx = b[G::x_off + slot(xrow, pc)];
      if constexpr (EPI == kEpiGrass) {
        // squares of bf16 values are exact in fp32; 8 of them summed in fp32,
        // then accumulated in fp64
        float s8 = 0.0f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float lo = bf_lo(bx[w]), hi = bf_hi(bx[w]);
          s8 = fmaf(lo, lo, s8);
          s8 = fmaf(hi, hi, s8);
        }
        sq += static_cast<double>(s8);
      }
      u32x4 be, bpv;
      if (HE) be = neg8(b[G::e_off + slot(erow, pc)]);
      if (HP && !kPT) bpv = neg8(b[G::p_off + slot(prow, pc)]);
#pragma unroll
      for (int t = 0; t < KT; ++t) {
        const u32x4 a = b[G::u_off + (j * KT + t) * 64 + lane];
        acc[t] = mfma(a, bx, acc[t]);
        if (HP && !kPT) acc[t] = mfma(a, bpv, acc[t]);
        if (HE) acc[t] = mfma(a, be, acc[t]);
      }
      if constexpr (kPT) {
#pragma unroll
        for (int jj = 0; jj < JPW; ++jj) {
          const int job = wave + jj * NW;  // wave-uniform
          if (job < NJOB) {
            const int pt = job / KT, t = job % KT;
            int r = 16 * pt + n;
            r = r < PR ? r : PR - 1;  // rows past the workgroup's are not used
            const u32x4 bp = neg8(b[G::p_off + slot(r, pc)]);
            pacc[jj] = mfma(b[G::u_off + (j * KT + t) * 64 + lane], bp, pacc[jj]);
          }
        }
      }
    }
  }
  if constexpr (kPT) {
    lds_barrier();  // every wave has read the last stage
    float *pu = reinterpret_cast<float *>(lds);  // PR x 16 KT floats in buffer 0
#pragma unroll
    for (int jj = 0; jj < JPW; ++jj) {
      const int job = wave + jj * NW;
      if (job < NJOB) {
        const int pt = job / KT, t = job % KT;
        const int r = 16 * pt + n;
        // lane (g, n) holds (-P U)[row r][16 t + 4 g .. + 3]
        if (r < PR) *reinterpret_cast<f32x4 *>(pu + r * (16 * KT) + 16 * t + 4 * g) = pacc[jj];
      }
    }
    lds_barrier();
#pragma unroll
    for (int t = 0; t < KT; ++t)
      acc[t] += *reinterpret_cast<const f32x4 *>(pu + prow * (16 * KT) + 16 * t + 4 * g);
  }

  // epilogue: lane (g, n) holds C[token, 16 t + 4 g .. +3]
  if constexpr (EPI == kEpiGrass) {
    // The row's loss term |g|^2 - |c|^2 + c D c^T (D = U^T U - I).  (D c)_a
    // on the matrix cores in fp32: A = fragments of D (staged once per
    // workgroup in LDS), B = the lane's own coefficients (contraction index
    // b = 16 t + 4 g + i of step (t, i)), so lane (g, n) receives (D c)_a of
    // token n for a = 16 at + 4 g + i, the same a as its acc[at][i]; D is
    // ~1e-3 in size, fp32 keeps the term to ~1e-7 of itself.  |c|^2 and the
    // sums in float64, the four lanes of a row and the workgroup's rows added
    // in a fixed order.  LDS after the last stage: the coefficients
    // [column][row of the workgroup] (for the operand), D's fragments, the
    // waves' loss sums.
    const int64_t Tg = T0 + wave;
    const bool ok = Tg < ntiles && 16 * Tg + n < tm.N;
    constexpr int RW = 16 * NW + 1;  // row stride in words: column reads spread over the banks
    constexpr int CT_W = (16 * KT * RW + 3) & ~3;
    constexpr int DF_W = KT * KT * 4 * 64;  // D fragments, [at][t][i][lane]
    static_assert((CT_W + DF_W) * 4 + NW * 8 <= NB * G::buf_units * 16, "epilogue exchange fits");
    float *cT = reinterpret_cast<float *>(lds);
    float *dl = cT + CT_W;
    double *wl = reinterpret_cast<double *>(dl + DF_W);
    lds_barrier();  // every wave is past its last stage
#pragma unroll
    for (int t = 0; t < KT; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) cT[(16 * t + 4 * g + i) * RW + 16 * wave + n] = ok ? acc[t][i] : 0.0f;
    // D[16 at + n'][16 t + 4 g' + i] for lane (g', n') of fragment (at, t, i)
    for (int e = wave * 64 + lane; e < DF_W; e += 64 * NW) {
      const int l2 = e & 63, f = e >> 6;
      const int i = f & 3, t = (f >> 2) % KT, at = (f >> 2) / KT;
      dl[e] = static_cast<float>(
          go.dgram[(16 * at + (l2 & 15)) * (16 * KT) + 16 * t + 4 * (l2 >> 4) + i]);
    }
    lds_barrier();
    double cc = 0.0;
    float q = 0.0f;
#pragma unroll
    for (int at = 0; at < KT; ++at) {
      f32x4 rr = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < KT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          rr = __builtin_amdgcn_mfma_f32_16x16x4f32(dl[((at * KT + t) * 4 + i) * 64 + lane],
                                                    acc[t][i], rr, 0, 0, 0);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        cc += static_cast<double>(acc[at][i]) * static_cast<double>(acc[at][i]);
        q = fmaf(acc[at][i], rr[i], q);
      }
    }
    sq += __shfl_xor(sq, 16, 64);
    sq += __shfl_xor(sq, 32, 64);
    cc += __shfl_xor(cc, 16, 64);
    cc += __shfl_xor(cc, 32, 64);
    q += __shfl_xor(q, 16, 64);
    q += __shfl_xor(q, 32, 64);
    double l = ok && g == 0 ? sq - cc + static_cast<double>(q) : 0.0;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) l += __shfl_xor(l, off, 64);
    if (lane == 0) wl[wave] = l;
    if (go.frag) {
      // slot (part p, 32-row step st of the workgroup, column tile t2, lane
      // 16 g2 + n2): rows 32 st + 8 g2 + 0..7 of operand column 16 t2 + n2 (of
      // 1 operand: C_hi for columns < k, C_lo of column - k below 2k; of 2:
      // part 0 C_hi, part 1 C_lo), zero past k and past row N
      constexpr int NST = NW / 2;
      const int ktb = go.ktb, nparts = go.nparts;
      const int64_t s_base = 16 * T0 / 32;
      const int64_t per_part = (go.npad / 32) * ktb * 64;
      const int nslots = nparts * NST * ktb * 64;
      for (int sl = wave * 64 + lane; sl < nslots; sl += 64 * NW) {
        const int p = sl / (NST * ktb * 64);
        const int rem = sl - p * (NST * ktb * 64);
        const int st = rem / (ktb * 64);
        const int t2 = (rem / 64) % ktb;
        const int l2 = rem & 63;
        const int g2 = l2 >> 4, n2 = l2 & 15;
        const int64_t c2 = 16 * t2 + n2;
        bool lo;
        int64_t col;
        if (nparts == 1) {
          lo = c2 >= k;
          col = lo ? c2 - k : c2;
        } else {
          lo = p == 1;
          col = c2;
        }
        const bool cvalid = col < k;
        uint32_t wd[4];
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
          bf16_t h[2];
#pragma unroll
          for (int e2 = 0; e2 < 2; ++e2) {
            const int row = 32 * st + 8 * g2 + 2 * qq + e2;
            const float x = cvalid ? cT[col * RW + row] : 0.0f;
            const bf16_t hi = from_f32<bf16_t>(x);
            h[e2] = lo ? from_f32<bf16_t>(x - to_f32(hi)) : hi;
          }
          wd[qq] = static_cast<uint32_t>(h[0]) | (static_cast<uint32_t>(h[1]) << 16);
        }
        const int64_t slot = p * per_part + ((s_base + st) * ktb + t2) * 64 + l2;
        *reinterpret_cast<u32x4 *>(reinterpret_cast<bf16_t *>(go.frag) + slot * 8) =
            u32x4{wd[0], wd[1], wd[2], wd[3]};
      }
    }
    lds_barrier();
    if (wave == 0 && lane == 0) {
      double tot = 0.0;
      for (int w2 = 0; w2 < NW; ++w2) tot += wl[w2];
      go.part[blockIdx.x] = tot;
    }
  }
  int64_t T = T0 + wave;
  if (T >= ntiles) return;  // a tile past the end computed a duplicate
  const int64_t i = 16 * T + n;
  const int64_t tok = tm.bp == 1 ? i : tile_token(tm, T, n);
  if (tm.bp == 1 && i >= tm.N) return;
  if (tok >= tm.N) return;  // a row past N of a short last sequence
  if constexpr (EPI == kEpiGrass) {
    if (!Cout) return;
  }
  if (EPI == kEpiProjected) {
    // C = X U - (P U)[pos] - (T_fixed U)[tok], in the paper's order
    if (pa.pu) {
      int64_t ps = pa.pos ? static_cast<int64_t>(pa.pos[tok]) : tok % pa.seq_len;
      ps = clamp_id(ps, pa.n_pos, pa.err_flag, 2);
      const float *pr = pa.pu + ps * pa.kp + 4 * g;
#pragma unroll
      for (int t = 0; t < KT; ++t) acc[t] -= *reinterpret_cast<const f32x4 *>(pr + 16 * t);
    }
    if (pa.eu) {
      const int64_t tk = clamp_id(pa.tok[tok], pa.vocab, pa.err_flag, 1);
      const float *er = pa.eu + tk * pa.kp + 4 * g;
#pragma unroll
      for (int t = 0; t < KT; ++t) acc[t] -= *reinterpret_cast<const f32x4 *>(er + 16 * t);
    }
  }
#pragma unroll
  for (int t = 0; t < KT; ++t) {
    const f32x4 v = acc[t];
    const int64_t j = 16 * t + 4 * g;
    if (EPI == kEpiF32) {  // full padded row of the projected table (columns >= k are 0)
      *reinterpret_cast<f32x4 *>(static_cast<float *>(Cout) + tok * ldc + j) = v;
      continue;
    }
    bf16_t *dst = static_cast<bf16_t *>(Cout) + tok * ldc + j;
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
// streaming compress: X U with no gathered rows
// ---------------------------------------------------------------------------
// Used for the gradient codec (no tables), for the projected-table compress
// (C = X U - (P U)[pos] - (T_fixed U)[tok], the subtraction done on the k
// coefficients of each token), and to build those projected tables.  A pure
// HBM stream of X is fastest when each compute wave issues its own loads:
// compute wave w owns 16 tokens and keeps D steps of its rows in flight in a
// register ring; the producer wave copies U chunk by chunk into two LDS
// buffers (one barrier per chunk).  The ring loads are unconditional (the
// loads past the end re-read the last step) and pinned in place, so the
// compiler keeps all D in flight.

template <int KT>
constexpr int s_chunk_steps() { return KT <= 4 ? 8 : 4; }

template <int KT, int EPI>
__global__ __launch_bounds__(kThreads) void stream_compress_kernel(
    const bf16_t *__restrict__ kfrag, int64_t d, int64_t k, const bf16_t *__restrict__ X,
    int64_t N, int64_t ldx, ProjArgs pa, void *__restrict__ Cout, int64_t ldc, int cvec) {
  constexpr int CH = s_chunk_steps<KT>();
  constexpr int D = CH;  // steps of rows in flight per wave
  constexpr int CHUNK_FRAGS = CH * KT;
  __shared__ u32x4 ubuf[2][CHUNK_FRAGS * 64];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int steps = static_cast<int>(d / 32);
  const int nchunks = (steps + CH - 1) / CH;
  const int rot = (steps % CH == 0) ? static_cast<int>(blockIdx.x % nchunks) * CH : 0;
  auto phys = [&](int si) { const int v = si + rot; return v >= steps ? v - steps : v; };

  if (wave == kW) {  // ------------------------------------------------ producer
    auto copy = [&](int cs) {
      const int c0 = phys(cs * CH) / CH;
      const int left = steps - c0 * CH;
      const int frags = (left < CH ? left : CH) * KT;
      dma_frags(kfrag + static_cast<int64_t>(c0) * CHUNK_FRAGS * 512, frags, ubuf[cs & 1], lane);
      wait_vmcnt<0>();
    };
    copy(0);
    lds_barrier();
    for (int cs = 0; cs < nchunks; ++cs) {
      if (cs + 1 < nchunks) copy(cs + 1);
      lds_barrier();
    }
    return;
  }

  const int g = lane >> 4, n = lane & 15;
  const int64_t tile = static_cast<int64_t>(blockIdx.x) * kW + wave;
  const int64_t it = 16 * tile + n;
  const int64_t i = it < N ? it : N - 1;  // padding lanes load token N-1 (not stored)
  const bf16_t *xr = X + i * ldx + 8 * g;

  f32x4 acc[KT];
#pragma unroll
  for (int t = 0; t < KT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto phys_c = [&](int si) { return phys(si < steps ? si : steps - 1); };
  u32x4 ring[D];
#pragma unroll
  for (int r = 0; r < D; ++r) ring[r] = ld16(xr + 32 * phys_c(r));

  const int nfull = steps / CH;
  for (int cs = 0; cs < nfull; ++cs) {
    lds_barrier();  // chunk cs is in ubuf[cs & 1]
    const u32x4 *ub = ubuf[cs & 1];
#pragma unroll
    for (int r = 0; r < CH; ++r) {
      const int si = cs * CH + r;
#pragma unroll
      for (int t = 0; t < KT; ++t) acc[t] = mfma(ub[(r * KT + t) * 64 + lane], ring[r % D], acc[t]);
      ring[r % D] = ld16(xr + 32 * phys_c(si + D));
      __builtin_amdgcn_sched_barrier(0);  // keep the refill here (see above)
    }
  }
  if (nfull < nchunks) {  // partial last chunk (no rotation in this case)
    lds_barrier();
    const u32x4 *ub = ubuf[nfull & 1];
#pragma unroll
    for (int r = 0; r < CH; ++r) {
      const int si = nfull * CH + r;
      if (si < steps) {
#pragma unroll
        for (int t = 0; t < KT; ++t)
          acc[t] = mfma(ub[(r * KT + t) * 64 + lane], ring[r % D], acc[t]);
      }
    }
  }
  lds_barrier();  // matches the producer's last barrier

  if (it >= N) return;
  if (EPI == kEpiProjected) {
    // C = X U - (P U)[pos] - (T_fixed U)[tok], in the paper's order
    if (pa.pu) {
      int64_t ps = pa.pos ? static_cast<int64_t>(pa.pos[it]) : it % pa.seq_len;
      ps = clamp_id(ps, pa.n_pos, pa.err_flag, 2);
      const float *pr = pa.pu + ps * pa.kp + 4 * g;
#pragma unroll
      for (int t = 0; t < KT; ++t) acc[t] -= *reinterpret_cast<const f32x4 *>(pr + 16 * t);
    }
    if (pa.eu) {
      const int64_t tk = clamp_id(pa.tok[it], pa.vocab, pa.err_flag, 1);
      const float *er = pa.eu + tk * pa.kp + 4 * g;
#pragma unroll
      for (int t = 0; t < KT; ++t) acc[t] -= *reinterpret_cast<const f32x4 *>(er + 16 * t);
    }
  }
#pragma unroll
  for (int t = 0; t < KT; ++t) {
    const f32x4 v = acc[t];
    const int64_t j = 16 * t + 4 * g;
    if (EPI == kEpiF32) {  // full padded row of the projected table (columns >= k are 0)
      *reinterpret_cast<f32x4 *>(static_cast<float *>(Cout) + it * ldc + j) = v;
      continue;
    }
    bf16_t *dst = static_cast<bf16_t *>(Cout) + it * ldc + j;
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

template <int KT, int EPI>
void launch_stream(const bf16_t *kf, const PackLayout &L, const void *X, int64_t N, int64_t ldx,
                   const ProjArgs &pa, void *C, int64_t ldc, int cvec, hipStream_t s) {
  dim3 grid(static_cast<unsigned>(ceil_div(ceil_div(N, 16), kW)));
  stream_compress_kernel<KT, EPI><<<grid, kThreads, 0, s>>>(
      kf, L.d, L.k, static_cast<const bf16_t *>(X), N, ldx, pa, C, ldc, cvec);
}

template <int EPI>
hipError_t launch_stream_kt(const PackLayout &L, const void *packed, const void *X, int64_t N,
                            int64_t ldx, const ProjArgs &pa, void *C, int64_t ldc, hipStream_t s) {
  const bf16_t *kf =
      reinterpret_cast<const bf16_t *>(static_cast<const char *>(packed) + L.off_kfrag);
  const int cvec = ((reinterpret_cast<uintptr_t>(C) & 7) == 0) && (ldc % 4 == 0);
  switch (L.kt) {
    case 1: launch_stream<1, EPI>(kf, L, X, N, ldx, pa, C, ldc, cvec, s); break;
    case 2: launch_stream<2, EPI>(kf, L, X, N, ldx, pa, C, ldc, cvec, s); break;
    case 3: launch_stream<3, EPI>(kf, L, X, N, ldx, pa, C, ldc, cvec, s); break;
    case 4: launch_stream<4, EPI>(kf, L, X, N, ldx, pa, C, ldc, cvec, s); break;
    case 5: launch_stream<5, EPI>(kf, L, X, N, ldx, pa, C, ldc, cvec, s); break;
    case 6: launch_stream<6, EPI>(kf, L, X, N, ldx, pa, C, ldc, cvec, s); break;
    case 7: launch_stream<7, EPI>(kf, L, X, N, ldx, pa, C, ldc, cvec, s); break;
    case 8: launch_stream<8, EPI>(kf, L, X, N, ldx, pa, C, ldc, cvec, s); break;
    default: return hipErrorNotSupported;
  }
  return hipGetLastError();
}

bool tables_ok(const IdArgs &ids) {
  if (ids.E && (!aligned16(ids.E) || ids.lde % 8 != 0)) return false;
  if (ids.P && (!aligned16(ids.P) || ids.ldp % 8 != 0)) return false;
  return true;
}

// Position-major tiling when the positions are the default i mod seq_len of a
// row-major [batch, seq_len] batch with batch a multiple of 4 (8 preferred)
// and whole workgroups of nw tiles.  The last sequence may be short by at
// most an eighth of a sequence: the tiles cover whole sequences and the
// missing rows are loaded (as token N - 1) but not stored.
bool pm_tiling_ok(int64_t N, const IdArgs &ids, int bp, int nw) {
  if (!ids.P || ids.pos || ids.seq_len <= 0 || N <= 0) return false;
  const int64_t seq = ids.seq_len;
  const int64_t batch = ceil_div(N, seq);
  if ((batch * seq - N) * 8 > seq) return false;
  // every workgroup holds nw full tiles: batch x seq / 16 must be a multiple of nw
  return batch % bp == 0 && seq % (16 / bp) == 0 && (batch * seq / 16) % nw == 0;
}

// Compute units of the current device (cached per device; concurrent first
// calls store the same value).
int device_cus() {
  static std::atomic<int> cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int c = cached[dev].load(std::memory_order_relaxed);
  if (c == 0) {
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        c <= 0)
      c = 256;
    cached[dev].store(c, std::memory_order_relaxed);
  }
  return c;
}

// Compute waves of a launch over N tokens: 8 where the stage buffers allow
// it and the launch still has a workgroup for every CU, else 4 (a launch of
// fewer, wider workgroups would leave CUs idle).
template <int KT, bool HE, bool HP, int BP>
int pick_nw(int64_t N) {
  if constexpr (nw_of<KT, HE, HP, BP>() != 8) {
    return 4;
  } else {
    return ceil_div(ceil_div(N, 16), 8) >= device_cus() ? 8 : 4;
  }
}

template <int KT, bool HE, bool HP, int BP, int EPI = kEpiBf16>
void launch_c(const bf16_t *kf, const PackLayout &L, const void *X, int64_t ldx, const Tiling &tm,
              const IdArgs &ids, void *C, int64_t ldc, int cvec, hipStream_t s,
              const ProjArgs &pa = ProjArgs{}, const GrassOut &go = GrassOut{}) {
  const int64_t ntiles = tile_count(tm);
  if constexpr (nw_of<KT, HE, HP, BP>() == 8) {
    if (pick_nw<KT, HE, HP, BP>(tm.N) == 8) {
      compress_kernel<KT, HE, HP, BP, 8, EPI>
          <<<dim3(static_cast<unsigned>(ceil_div(ntiles, 8))), threads_c<8>(), 0, s>>>(
              kf, L.d, L.k, static_cast<const bf16_t *>(X), ldx, tm, ids, pa, C, ldc, cvec, go);
      return;
    }
  }
  compress_kernel<KT, HE, HP, BP, 4, EPI>
      <<<dim3(static_cast<unsigned>(ceil_div(ntiles, 4))), threads_c<4>(), 0, s>>>(
          kf, L.d, L.k, static_cast<const bf16_t *>(X), ldx, tm, ids, pa, C, ldc, cvec, go);
}

// X U with no gathered rows, on the staged kernel (d a multiple of kStageCols)
template <int EPI>
hipError_t launch_plain_kt(const PackLayout &L, const void *packed, const void *X, int64_t N,
                           int64_t ldx, const ProjArgs &pa, void *C, int64_t ldc, hipStream_t s) {
  const bf16_t *kf =
      reinterpret_cast<const bf16_t *>(static_cast<const char *>(packed) + L.off_kfrag);
  const int cvec = ((reinterpret_cast<uintptr_t>(C) & 7) == 0) && (ldc % 4 == 0);
  const Tiling tm{N, 1, 1};
  const IdArgs none{};
  switch (L.kt) {
    case 1: launch_c<1, false, false, 1, EPI>(kf, L, X, ldx, tm, none, C, ldc, cvec, s, pa); break;
    case 2: launch_c<2, false, false, 1, EPI>(kf, L, X, ldx, tm, none, C, ldc, cvec, s, pa); break;
    case 3: launch_c<3, false, false, 1, EPI>(kf, L, X, ldx, tm, none, C, ldc, cvec, s, pa); break;
    case 4: launch_c<4, false, false, 1, EPI>(kf, L, X, ldx, tm, none, C, ldc, cvec, s, pa); break;
    case 5: launch_c<5, false, false, 1, EPI>(kf, L, X, ldx, tm, none, C, ldc, cvec, s, pa); break;
    case 6: launch_c<6, false, false, 1, EPI>(kf, L, X, ldx, tm, none, C, ldc, cvec, s, pa); break;
    case 7: launch_c<7, false, false, 1, EPI>(kf, L, X, ldx, tm, none, C, ldc, cvec, s, pa); break;
    case 8: launch_c<8, false, false, 1, EPI>(kf, L, X, ldx, tm, none, C, ldc, cvec, s, pa); break;
    default: return hipErrorNotSupported;
  }
  return hipGetLastError();
}

// X U with no gathered rows: the staged kernel when d allows, else the
// register-ring streaming kernel
template <int EPI>
hipError_t launch_plain(const PackLayout &L, const void *packed, const void *X, int64_t N,
                        int64_t ldx, const ProjArgs &pa, void *C, int64_t ldc, hipStream_t s) {
  if (L.d % kStageCols == 0) return launch_plain_kt<EPI>(L, packed, X, N, ldx, pa, C, ldc, s);
  return launch_stream_kt<EPI>(L, packed, X, N, ldx, pa, C, ldc, s);
}

template <int KT>
void launch_c_kt(const bf16_t *kf, const PackLayout &L, const void *X, int64_t ldx,
                 const Tiling &tm, const IdArgs &ids, void *C, int64_t ldc, int cvec,
                 hipStream_t s) {
  const bool he = ids.E != nullptr, hp = ids.P != nullptr;
  const int64_t N = tm.N;
  // position-major tiles (8 batches per tile, else 4) when whole workgroups
  // of tiles allow them
  const Tiling tm8{N, ids.seq_len, 8, 0}, tm4{N, ids.seq_len, 4, 0};
  if (he && hp) {
    // Each P row is read once per call; beside T_fixed a large P (over
    // 64 MiB) would evict the T_fixed rows that repeated ids reuse, so its
    // rows are copied non-temporally.  A small P is kept in the caches.
    const int ps = ids.n_pos * L.d * 2 > (int64_t{64} << 20) ? 1 : 0;
    const Tiling s8{N, ids.seq_len, 8, ps}, s4{N, ids.seq_len, 4, ps}, s1{N, 1, 1, ps};
    if (pm_tiling_ok(N, ids, 8, pick_nw<KT, true, true, 8>(N)))
      launch_c<KT, true, true, 8>(kf, L, X, ldx, s8, ids, C, ldc, cvec, s);
    else if (pm_tiling_ok(N, ids, 4, pick_nw<KT, true, true, 4>(N)))
      launch_c<KT, true, true, 4>(kf, L, X, ldx, s4, ids, C, ldc, cvec, s);
    else
      launch_c<KT, true, true, 1>(kf, L, X, ldx, s1, ids, C, ldc, cvec, s);
  } else if (he) {
    launch_c<KT, true, false, 1>(kf, L, X, ldx, tm, ids, C, ldc, cvec, s);
  } else {
    if (pm_tiling_ok(N, ids, 8, pick_nw<KT, false, true, 8>(N)))
      launch_c<KT, false, true, 8>(kf, L, X, ldx, tm8, ids, C, ldc, cvec, s);
    else if (pm_tiling_ok(N, ids, 4, pick_nw<KT, false, true, 4>(N)))
      launch_c<KT, false, true, 4>(kf, L, X, ldx, tm4, ids, C, ldc, cvec, s);
    else
      launch_c<KT, false, true, 1>(kf, L, X, ldx, tm, ids, C, ldc, cvec, s);
  }
}

}  // namespace

bool compress_mfma_ok(const PackLayout &L, const void *X, int64_t ldx, const IdArgs &ids) {
  if (!ids.E && !ids.P) return stream_mfma_ok(L, X, ldx);
  return L.mfma && L.d % kStageCols == 0 && aligned16(X) && ldx % 8 == 0 && tables_ok(ids);
}

hipError_t launch_compress_mfma(const PackLayout &L, const void *packed, const void *X,
                                int64_t N, int64_t ldx, const IdArgs &ids, void *C, int64_t ldc,
                                hipStream_t s) {
  const bf16_t *kf =
      reinterpret_cast<const bf16_t *>(static_cast<const char *>(packed) + L.off_kfrag);
  const int cvec = ((reinterpret_cast<uintptr_t>(C) & 7) == 0) && (ldc % 4 == 0);
  if (!ids.E && !ids.P) return launch_plain<kEpiBf16>(L, packed, X, N, ldx, ProjArgs{}, C, ldc, s);
  const Tiling tm{N, 1, 1};  // token-major; the table dispatch picks position-major tiles
  switch (L.kt) {
    case 1: launch_c_kt<1>(kf, L, X, ldx, tm, ids, C, ldc, cvec, s); break;
    case 2: launch_c_kt<2>(kf, L, X, ldx, tm, ids, C, ldc, cvec, s); break;
    case 3: launch_c_kt<3>(kf, L, X, ldx, tm, ids, C, ldc, cvec, s); break;
    case 4: launch_c_kt<4>(kf, L, X, ldx, tm, ids, C, ldc, cvec, s); break;
    case 5: launch_c_kt<5>(kf, L, X, ldx, tm, ids, C, ldc, cvec, s); break;
    case 6: launch_c_kt<6>(kf, L, X, ldx, tm, ids, C, ldc, cvec, s); break;
    case 7: launch_c_kt<7>(kf, L, X, ldx, tm, ids, C, ldc, cvec, s); break;
    case 8: launch_c_kt<8>(kf, L, X, ldx, tm, ids, C, ldc, cvec, s); break;
    default: return hipErrorNotSupported;
  }
  return hipGetLastError();
}

bool stream_mfma_ok(const PackLayout &L, const void *X, int64_t ldx) {
  return L.mfma && aligned16(X) && ldx % 8 == 0;
}

hipError_t launch_table_project_mfma(const PackLayout &L, const void *packed, const void *T,
                                     int64_t rows, int64_t ldt, float *out, int64_t kp,
                                     hipStream_t s) {
  return launch_plain<kEpiF32>(L, packed, T, rows, ldt, ProjArgs{}, out, kp, s);
}

hipError_t launch_compress_projected_mfma(const PackLayout &L, const void *packed, const void *X,
                                          int64_t N, int64_t ldx, const ProjArgs &pa, void *C,
                                          int64_t ldc, hipStream_t s) {
  return launch_plain<kEpiProjected>(L, packed, X, N, ldx, pa, C, ldc, s);
}

int64_t grass_compress_groups(const PackLayout &L, int64_t N, int64_t *steps) {
  int nw = 4;
  switch (L.kt) {
    case 1: nw = pick_nw<1, false, false, 1>(N); break;
    case 2: nw = pick_nw<2, false, false, 1>(N); break;
    case 3: nw = pick_nw<3, false, false, 1>(N); break;
    case 4: nw = pick_nw<4, false, false, 1>(N); break;
    case 5: nw = pick_nw<5, false, false, 1>(N); break;
    case 6: nw = pick_nw<6, false, false, 1>(N); break;
    case 7: nw = pick_nw<7, false, false, 1>(N); break;
    case 8: nw = pick_nw<8, false, false, 1>(N); break;
    default: break;
  }
  const int64_t groups = ceil_div(ceil_div(N, 16), nw);
  if (steps) *steps = groups * (nw / 2);
  return groups;
}

hipError_t launch_grass_compress_mfma(const PackLayout &L, const void *packed, const void *G,
                                      int64_t N, int64_t ldg, const GrassOut &go, void *Cwire,
                                      int64_t ldc, hipStream_t s) {
  if (!L.mfma || L.d % kStageCols != 0) return hipErrorNotSupported;
  const bf16_t *kf =
      reinterpret_cast<const bf16_t *>(static_cast<const char *>(packed) + L.off_kfrag);
  const int cvec = Cwire && ((reinterpret_cast<uintptr_t>(Cwire) & 7) == 0) && (ldc % 4 == 0);
  const Tiling tm{N, 1, 1};
  const IdArgs none{};
  const ProjArgs pa{};
  switch (L.kt) {
    case 1: launch_c<1, false, false, 1, kEpiGrass>(kf, L, G, ldg, tm, none, Cwire, ldc, cvec, s, pa, go); break;
    case 2: launch_c<2, false, false, 1, kEpiGrass>(kf, L, G, ldg, tm, none, Cwire, ldc, cvec, s, pa, go); break;
    case 3: launch_c<3, false, false, 1, kEpiGrass>(kf, L, G, ldg, tm, none, Cwire, ldc, cvec, s, pa, go); break;
    case 4: launch_c<4, false, false, 1, kEpiGrass>(kf, L, G, ldg, tm, none, Cwire, ldc, cvec, s, pa, go); break;
    case 5: launch_c<5, false, false, 1, kEpiGrass>(kf, L, G, ldg, tm, none, Cwire, ldc, cvec, s, pa, go); break;
    case 6: launch_c<6, false, false, 1, kEpiGrass>(kf, L, G, ldg, tm, none, Cwire, ldc, cvec, s, pa, go); break;
    case 7: launch_c<7, false, false, 1, kEpiGrass>(kf, L, G, ldg, tm, none, Cwire, ldc, cvec, s, pa, go); break;
    case 8: launch_c<8, false, false, 1, kEpiGrass>(kf, L, G, ldg, tm, none, Cwire, ldc, cvec, s, pa, go); break;
    default: return hipErrorNotSupported;
  }
  return hipGetLastError();
}

}  // namespace sn
