// Matrix-core decompress: X[i, :] = C[i, :] U^T + P[pos_i, :] + T_fixed[tok[i], :]
// (Sec. 4.3.1; with no tables, the gradient recovery Cg U^T of Sec. 4.4).
//
// Work split: a workgroup owns one 256-column block of X and a run of
// 16-token tiles; consecutive workgroups take consecutive token runs of the
// same column block.  The block's slice of U (rfrag layout, 8 row groups of
// 32 columns) is copied into LDS once and stays there, so the main loop has
// no barriers: every wave walks its own tiles.
//
// Per tile and 128-column chunk a wave
//  1. runs 4 row groups x 2 x ceil(k/32) MFMAs (A = U fragment from LDS,
//     B = the tile's coefficients); lane (g, n) gets 8 consecutive columns
//     of token n in fp32;
//  2. passes the fp32 tile through a wave-private LDS buffer to the row
//     layout in which every memory instruction covers 4 rows x 256
//     contiguous bytes (lane (q, m): rows 4 i + q, columns 8 m .. 8 m + 7);
//  3. adds the P and T_fixed values of those columns, loaded one chunk ahead
//     in the same row layout (both tables: one bf16 dot-product instruction
//     per value), rounds once to bf16 and stores 16 bytes.
// Contiguous 256-byte row pieces are the cheapest pattern for both the
// gathers and the stores; the MFMA operand layout (16 rows x 64 bytes per
// instruction) is markedly slower for both.
#include "sn_mfma_common.h"

namespace sn {
namespace {

constexpr int kDW = 4;              // waves per workgroup
constexpr int kDThreads = 64 * kDW;
constexpr int kPG = 8;              // 32-column row groups per column block (256 columns)
constexpr int kDCols = 32 * kPG;    // columns per block
constexpr int kNC = kPG / 4;        // 128-column chunks per block
constexpr int kMaxWaveTiles = 16;   // tiles per wave (ids staged in LDS)

struct DTiling {
  int N;           // tokens (< 2^31)
  int seq, batch;  // position-major tile order when batch > 0
};

// First token of tile T and, in position-major order, its first position:
// the batch index varies fastest, so neighbouring tiles share positional rows.
__device__ __forceinline__ int dtile_token0(const DTiling &tm, unsigned T) {
  if (tm.batch > 0) return static_cast<int>((T % tm.batch) * tm.seq + (T / tm.batch) * 16);
  return static_cast<int>(16 * T);
}
__device__ __forceinline__ int dtile_pos0(const DTiling &tm, unsigned T) {
  return static_cast<int>((T / tm.batch) * 16);
}

// Out-of-range id: clamp it into the table and remember the flag bit.
__device__ __forceinline__ int64_t clamp_flag(int64_t id, int64_t rows, int bit, int &bad) {
  bad |= (id < 0 || id >= rows) ? bit : 0;
  return id < 0 ? 0 : (id >= rows ? rows - 1 : id);
}

// 16-byte slot of (row r, 4-float unit u) in a wave's 16 x 128 fp32 tile.
// Units 2m and 2m+1 (the 8 columns lane m reads back) are split into the two
// halves of the row and the position is XORed with the row, so both the
// MFMA-layout writes (16 rows, one unit) and the row-layout reads (one row,
// 16 units) touch 16 distinct bank groups.
__device__ __forceinline__ int ot_slot(int r, int u) {
  return r * 32 + (((u >> 1) | ((u & 1) << 4)) ^ (r & 15));
}

// Per-tile state of a lane: the MFMA B operand (coefficients of token n) and,
// for its 4 rows 4 i + q of the row layout, the token, T_fixed row and P row
// (row indices, not pointers: 32-bit registers).
template <int KS>
struct DTile {
  u32x4 b[KS];
  int er[4], pr[4], xr[4];
};

template <int KS, int CM>
__device__ __forceinline__ void load_coeffs(DTile<KS> &dt, int t, const bf16_t *__restrict__ C,
                                            int64_t ldc, int64_t k, int g) {
  // C[t, 32 q + 8 g + e].  U's fragments are zero past column k, so a lane
  // whose columns lie past k may load any finite values: it loads the row's
  // first columns instead, with no branch and no select, and the values are
  // first touched by the MFMA.
  const bf16_t *cr = C + static_cast<int64_t>(t) * ldc;
#pragma unroll
  for (int q = 0; q < KS; ++q) {
    const int64_t c0 = 32 * q + 8 * g;
    if (CM == 0) {  // 16-byte rows, k % 8 == 0: a chunk is all in or all out
      dt.b[q] = ld16(cr + (c0 < k ? c0 : 0));
    } else if (CM == 1) {  // 4-byte rows, k even: pairs are all in or all out
      const uint32_t *cw = reinterpret_cast<const uint32_t *>(cr);
      uint32_t w[4];
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        const int64_t j = c0 + 2 * e2;
        w[e2] = cw[(j < k ? j : 0) / 2];
      }
      dt.b[q] = u32x4{w[0], w[1], w[2], w[3]};
    } else {
      uint32_t w[4];
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        const int64_t j0 = c0 + 2 * e2, j1 = j0 + 1;
        w[e2] = static_cast<uint32_t>(cr[j0 < k ? j0 : 0]) |
                (static_cast<uint32_t>(cr[j1 < k ? j1 : 0]) << 16);
      }
      dt.b[q] = u32x4{w[0], w[1], w[2], w[3]};
    }
  }
}

// Gathered values in the row layout (rows 4 i + q): T_fixed for both chunks
// of a tile, P for one chunk.
struct ERows {
  u32x4 v[kNC][4];
};
struct PRows {
  u32x4 v[4];
};

__device__ __forceinline__ void add8(float (&o)[8], u32x4 v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    o[2 * e] += bf_lo(w[e]);
    o[2 * e + 1] += bf_hi(w[e]);
  }
}

// o[j] += T_fixed[j] + P[j] for the 8 values of two 16-byte row pieces: the
// (T_fixed, P) pair of column j is packed into one dword and added to o[j] by
// the bf16 dot-product instruction with weights (1, 1), one instruction per
// value instead of two conversions and two adds.  The instruction aligns its
// three addends itself and is not correctly rounded; on 4M random triples
// spread over 20 binades (cancelling pairs included) its error stayed within
// 2.25 units in the last place of the largest addend, against 2.75 for two
// fp32 adds, so the bf16 result is as accurate as with the adds.
__device__ __forceinline__ void add8_ep(float (&o)[8], u32x4 e, u32x4 p) {
  const uint32_t we[4] = {e.x, e.y, e.z, e.w}, wp[4] = {p.x, p.y, p.z, p.w};
  const bf16x2 one = __builtin_bit_cast(bf16x2, 0x3f803f80u);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bf16x2 lo = __builtin_bit_cast(bf16x2, __builtin_amdgcn_perm(we[i], wp[i], 0x01000504u));
    const bf16x2 hi = __builtin_bit_cast(bf16x2, __builtin_amdgcn_perm(we[i], wp[i], 0x03020706u));
    o[2 * i] = __builtin_amdgcn_fdot2_f32_bf16(lo, one, o[2 * i], false);
    o[2 * i + 1] = __builtin_amdgcn_fdot2_f32_bf16(hi, one, o[2 * i + 1], false);
  }
}

// LDS of a workgroup besides the U slice: the per-wave transpose buffers
// (32 KiB; with the 48 KiB slice at ks = 3, two workgroups fill a CU's 160 KiB).
struct DSmem {
  f32x4 ot[kDW][16 * 32];
};

// PS: load the P rows with non-temporal loads (each is read once per call).
template <int KS, bool HE, bool HP, int CM, bool PS>
__global__ __launch_bounds__(kDThreads) void decompress_cb_kernel(
    const bf16_t *__restrict__ rfrag, int64_t k, const bf16_t *__restrict__ C, int64_t ldc,
    DTiling tm, IdArgs ids, ColSegs xs, int ncb, int ntiles,
    int tiles_per_wg, int young_from) {
  constexpr int FR = 2 * KS;  // fragments per row group
  __shared__ u32x4 us[kPG * FR * 64];
  constexpr bool kIds = HE || HP;
  __shared__ DSmem sm;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // Column block = workgroup index mod the number of blocks: workgroups are
  // dealt to the 8 XCDs round robin, so each XCD (and its L2) sees only the
  // columns of ncb / 8 blocks, of U, T_fixed and P alike.
  const int cb = static_cast<int>(blockIdx.x % static_cast<unsigned>(ncb));
  const int tg = static_cast<int>(blockIdx.x / static_cast<unsigned>(ncb));
  const int g = lane >> 4, n = lane & 15;  // MFMA layout
  const int q = lane >> 4, m = lane & 15;  // row layout

  // each wave takes a contiguous run of the workgroup's tiles
  const int per_wave = tiles_per_wg / kDW;
  const int T0 = tg * tiles_per_wg + wave * per_wave;
  const int T1 = T0 + per_wave < ntiles ? T0 + per_wave : ntiles;
  const int nt = T0 < T1 ? T1 - T0 : 0;  // this wave's tiles

  // Token of row r of the wave's j-th tile (clamped to the wave's last tile).
  // Rows past the last token read the rows of token N-1 (every load stays in
  // bounds).  Without P they compute and store exactly the bytes of row N-1
  // again (unconditional stores); with P they are not stored, since in
  // position-major order they may reuse another sequence's positional rows.
  auto tile_of = [&](int j) { return static_cast<unsigned>(T0 + (j < nt ? j : nt - 1)); };
  auto token = [&](unsigned T, int r) {
    const int t = dtile_token0(tm, T) + r;
    return t < tm.N ? t : tm.N - 1;
  };

  // Load the ids of all the wave's tiles up front (fixed trip count, clamped
  // tiles: all loads are in flight before the first wait) and clamp each into
  // its table (out-of-range ids set a flag bit).  They stay in registers:
  // lane (g, n) holds row n of tiles 4 i + g in entry i, and the lanes that need
  // a row fetch it with a cross-lane permute (no LDS allocation, so the
  // tables cost no occupancy).
  int bad = 0;
  static_assert(kMaxWaveTiles == 16, "four entries per lane");
  // token ids e0..e3 and position ids q0..q3: plain scalars, never indexed
  int e0 = 0, e1 = 0, e2 = 0, e3 = 0, q0 = 0, q1 = 0, q2 = 0, q3 = 0;
  if constexpr (kIds) {
    if (nt > 0) {
      auto tok_id = [&](int i) {
        return HE ? ids.tok[token(tile_of(4 * i + g), n)] : 0;
      };
      auto pos_id = [&](int i) {
        if (!HP) return 0;
        const unsigned T = tile_of(4 * i + g);
        const int t = token(T, n);
        if (ids.pos) return ids.pos[t];
        if (tm.batch > 0 && dtile_token0(tm, T) + n < tm.N) return dtile_pos0(tm, T) + n;
        // token-major order, or a row past N (its clamped token's position)
        return static_cast<int>(static_cast<unsigned>(t) % static_cast<unsigned>(ids.seq_len));
      };
      e0 = tok_id(0); e1 = tok_id(1); e2 = tok_id(2); e3 = tok_id(3);
      q0 = pos_id(0); q1 = pos_id(1); q2 = pos_id(2); q3 = pos_id(3);
      auto ce = [&](int id) {
        return HE ? static_cast<int>(clamp_flag(id, ids.vocab, 1, bad)) : 0;
      };
      auto cp = [&](int id) {
        return HP ? static_cast<int>(clamp_flag(id, ids.n_pos, 2, bad)) : 0;
      };
      e0 = ce(e0); e1 = ce(e1); e2 = ce(e2); e3 = ce(e3);
      q0 = cp(q0); q1 = cp(q1); q2 = cp(q2); q3 = cp(q3);
    }
  }
  {  // the block's U slice -> LDS, 1 KiB per direct-to-LDS load
    const bf16_t *src = rfrag + static_cast<int64_t>(cb) * kPG * FR * 512;
    for (int f = wave; f < kPG * FR; f += kDW) lds_dma_16(src + f * 512 + lane * 8, us + f * 64);
    wait_vmcnt<0>();
  }
  __syncthreads();
  if (nt == 0) return;

  const int64_t col_r = static_cast<int64_t>(cb) * kDCols + 8 * m;  // row-layout column
  // the column segment of X that holds this block (blocks never straddle two)
  int sg = 0;
  while (sg + 1 < xs.n && static_cast<int64_t>(cb) * kDCols >= xs.c0[sg + 1]) ++sg;
  // Row addresses are base + row x row-bytes with both factors below 2^32
  // (the launch checks the leading dimensions): one 32 x 32 -> 64-bit
  // multiply-add per row, no 64-bit products.
  const uint32_t ldx_b = static_cast<uint32_t>(xs.ld[sg] * 2);
  f32x4 *otw = sm.ot[wave];

  auto load_tile = [&](DTile<KS> &dt, int j) {
    const unsigned T = tile_of(j);
    const int t0 = dtile_token0(tm, T);  // the tile's first token, once per tile
    auto tok_of = [&](int r) { return t0 + r < tm.N ? t0 + r : tm.N - 1; };
    load_coeffs<KS, CM>(dt, tok_of(n), C, ldc, k, g);
    // Tiles are loaded in order 0, 1, 2, ...: every fourth tile the entries
    // move down one, so tile j's ids are always in entry 0 (a wave-uniform
    // branch and register moves; a choice among the entries by j / 4 would be
    // compiled to an indexed access to private memory).  Past the last tile
    // (j >= nt) entry 0 holds ids of the last staged tiles: valid rows, and
    // the repeated tile is never stored.
    if (j > 0 && (j & 3) == 0) {
      e0 = e1; e1 = e2; e2 = e3;
      q0 = q1; q1 = q2; q2 = q3;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 4 * i + q;
      if constexpr (kIds) {  // row r of tile j: lane 16 (j % 4) + r, entry 0
        const int src = (16 * (j & 3) + r) * 4;
        if (HE) dt.er[i] = __builtin_amdgcn_ds_bpermute(src, e0);
        if (HP) dt.pr[i] = __builtin_amdgcn_ds_bpermute(src, q0);
      }
      if constexpr (HP)
        dt.xr[i] = t0 + r < tm.N ? t0 + r : -1;  // -1: past N, not stored
      else
        dt.xr[i] = tok_of(r);
    }
  };
  const char *Eb = reinterpret_cast<const char *>(static_cast<const bf16_t *>(ids.E) + col_r);
  const char *Pb = reinterpret_cast<const char *>(static_cast<const bf16_t *>(ids.P) + col_r);
  char *Xb = reinterpret_cast<char *>(static_cast<bf16_t *>(xs.base[sg]) + (col_r - xs.c0[sg]));
  const uint32_t lde_b = static_cast<uint32_t>(ids.lde * 2);
  const uint32_t ldp_b = static_cast<uint32_t>(ids.ldp * 2);
  auto row_at = [](const char *base, int row, uint32_t ld_b) {
    return reinterpret_cast<const bf16_t *>(
        base + static_cast<uint64_t>(static_cast<uint32_t>(row)) * ld_b);
  };
  // T_fixed values are loaded a whole tile ahead (double buffer).  P values
  // are reloaded only when the tile's positions change: in position-major
  // order a wave's run of tiles holds `batch` tiles with the same 16
  // positions in a row; chunk c's P values are refilled right after chunk c
  // of the previous tile has used them.
  auto load_e = [&](ERows &er, const DTile<KS> &dt) {
#pragma unroll
    for (int c = 0; c < kNC; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        er.v[c][i] = ld16(row_at(Eb, dt.er[i], lde_b) + 128 * c);
  };
  auto load_p = [&](PRows &pr, const DTile<KS> &dt, int c) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bf16_t *src = row_at(Pb, dt.pr[i], ldp_b) + 128 * c;
      if constexpr (PS)
        pr.v[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(src));
      else
        pr.v[i] = ld16(src);
    }
  };
  // whether tile j has other positions than tile j - 1 (always, unless position-major)
  auto new_pos = [&](int j) {
    if (tm.batch == 0 || j == 0) return true;
    return tile_of(j) / static_cast<unsigned>(tm.batch) !=
           tile_of(j - 1) / static_cast<unsigned>(tm.batch);
  };

  // one chunk: MFMAs, transpose through LDS, add the gathered rows, store
  auto chunk = [&](const DTile<KS> &dt, int c, const ERows &er, const PRows &pr) {
    f32x4 acc[4][2];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int pg = 4 * c + p;
      acc[p][0] = f32x4{0.f, 0.f, 0.f, 0.f};
      acc[p][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int qq = 0; qq < KS; ++qq) {
        acc[p][0] = mfma(us[((pg * 2 + 0) * KS + qq) * 64 + lane], dt.b[qq], acc[p][0]);
        acc[p][1] = mfma(us[((pg * 2 + 1) * KS + qq) * 64 + lane], dt.b[qq], acc[p][1]);
      }
    }
    // lane (g, n): token n, columns 32 p + 8 g + 4 h + 0..3 = unit 8 p + 2 g + h
#pragma unroll
    for (int p = 0; p < 4; ++p)
#pragma unroll
      for (int h = 0; h < 2; ++h) otw[ot_slot(n, 8 * p + 2 * g + h)] = acc[p][h];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 4 * i + q;
      const f32x4 lo = otw[ot_slot(r, 2 * m)], hi = otw[ot_slot(r, 2 * m + 1)];
      float o[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      if (HP && HE) {
        add8_ep(o, er.v[c][i], pr.v[i]);
      } else {
        if (HP) add8(o, pr.v[i]);
        if (HE) add8(o, er.v[c][i]);
      }
      // Non-temporal store: X is written once and not read back here, and
      // keeping it out of the caches leaves L2 to the gathered rows (the
      // gathers' hit rate, and with it the kernel time, depends on it).
      if (!HP || dt.xr[i] >= 0)
        __builtin_nontemporal_store(
            u32x4{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]), pack_bf16x2(o[4], o[5]),
                  pack_bf16x2(o[6], o[7])},
            reinterpret_cast<u32x4 *>(const_cast<bf16_t *>(row_at(Xb, dt.xr[i], ldx_b)) +
                                      128 * c));
    }
  };

  static_assert(kNC == 2, "two chunks per block");
  DTile<KS> cur, nxt;
  ERows eA, eB;
  PRows p0, p1;
  load_tile(cur, 0);
  if (HE) load_e(eA, cur);
  if (HP) {
    load_p(p0, cur, 0);
    load_p(p1, cur, 1);
  }
  // tile j: its T_fixed values are in ec, the next tile's go to en
  auto tile_step = [&](int j, ERows &ec, ERows &en) {
    // Keep the U fragments in LDS: without this the compiler would hoist
    // every fragment read out of the loop into registers and halve the
    // number of resident waves.
    asm volatile("" ::: "memory");
    load_tile(nxt, j + 1);  // the last tile repeats itself
    if (HE) load_e(en, nxt);
    const bool np1 = HP && j + 1 < nt && new_pos(j + 1);
    chunk(cur, 0, ec, p0);
    if (np1) load_p(p0, nxt, 0);
    chunk(cur, 1, ec, p1);
    if (np1) load_p(p1, nxt, 1);
    cur = nxt;
  };
  // The workgroups dispatched after every CU has one (the second on a CU)
  // lose issue arbitration to the older waves on the same SIMDs and would
  // end ~5 us later; their waves run at raised priority for the first half
  // of their tiles, then at the default (pair at d = 4096: 131.1 -> 129.6 us).
  const bool young = static_cast<int>(blockIdx.x) >= young_from;
  if (young) __builtin_amdgcn_s_setprio(2);
  for (int j = 0; j < nt; j += 2) {
    if (young && j == nt / 2) __builtin_amdgcn_s_setprio(0);
    tile_step(j, eA, eB);
    if (j + 1 < nt) tile_step(j + 1, eB, eA);
  }
  if (bad && ids.err_flag) atomicOr(ids.err_flag, bad);
}

// Resident workgroups of a kernel on the current device (CUs x occupancy)
// and the CUs.
struct Slots {
  int64_t slots, cus;
};
template <typename K>
Slots resident_slots(K kernel) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(kernel),
                                                   kDThreads, 0) != hipSuccess ||
      cus <= 0 || per_cu <= 0)
    return Slots{512, 256};
  return Slots{static_cast<int64_t>(cus) * per_cu, cus};
}

template <int KS, bool HE, bool HP, int CM, bool PS = false>
void launch_dcb(const bf16_t *rf, const PackLayout &L, const void *C, int64_t ldc,
                const DTiling &tm, const IdArgs &ids, const ColSegs &X, hipStream_t s) {
  const int ncb = static_cast<int>(L.d / kDCols);
  // position-major tiles cover whole [batch, seq] sequences (the last one may
  // be short: its missing rows are read but not stored)
  const int64_t ntiles = tm.batch > 0 ? static_cast<int64_t>(tm.batch) * (tm.seq / 16)
                                      : ceil_div(tm.N, 16);
  // one round of resident workgroups over the whole grid, whole waves of tiles
  static const Slots sl = resident_slots(decompress_cb_kernel<KS, HE, HP, CM, PS>);
  const int64_t groups = sl.slots / ncb > 0 ? sl.slots / ncb : 1;  // token groups per round
  int64_t per = ceil_div(ntiles, groups);
  per = per < kDW ? kDW : (per > kDW * kMaxWaveTiles ? kDW * kMaxWaveTiles : per);
  per = ceil_div(per, kDW) * kDW;
  const int64_t tgroups = ceil_div(ntiles, per);
  dim3 grid(static_cast<unsigned>(tgroups * ncb));
  // workgroups past the first one per CU (when the grid has more)
  const int64_t young_from = tgroups * ncb > sl.cus ? sl.cus : tgroups * ncb;
  decompress_cb_kernel<KS, HE, HP, CM, PS><<<grid, kDThreads, 0, s>>>(
      rf, L.k, static_cast<const bf16_t *>(C), ldc, tm, ids, X, ncb,
      static_cast<int>(ntiles), static_cast<int>(per), static_cast<int>(young_from));
}

template <int KS, int CM>
void launch_dcb_t(const bf16_t *rf, const PackLayout &L, const void *C, int64_t ldc,
                  const DTiling &tm, const IdArgs &ids, const ColSegs &X, hipStream_t s) {
  const bool he = ids.E != nullptr, hp = ids.P != nullptr;
  // Each P row piece is read once per call.  Beside T_fixed, a large P
  // (over 64 MiB) streams through the caches and evicts the T_fixed rows that
  // are reused: it is loaded non-temporally (d = 8192: ~235 -> ~200 us at
  // 32768 tokens).  Alone, or when small, it is loaded normally and stays in
  // the 256 MB Infinity Cache from one call to the next.
  if (he && hp && ids.n_pos * L.d * 2 > (int64_t{64} << 20))
    launch_dcb<KS, true, true, CM, true>(rf, L, C, ldc, tm, ids, X, s);
  else if (he && hp)
    launch_dcb<KS, true, true, CM>(rf, L, C, ldc, tm, ids, X, s);
  else if (he)
    launch_dcb<KS, true, false, CM>(rf, L, C, ldc, tm, ids, X, s);
  else if (hp)
    launch_dcb<KS, false, true, CM>(rf, L, C, ldc, tm, ids, X, s);
  else
    launch_dcb<KS, false, false, CM>(rf, L, C, ldc, tm, ids, X, s);
}

template <int KS>
void launch_dcb_ks(const bf16_t *rf, const PackLayout &L, const void *C, int64_t ldc, int cmode,
                   const DTiling &tm, const IdArgs &ids, const ColSegs &X, hipStream_t s) {
  if (cmode == 0)
    launch_dcb_t<KS, 0>(rf, L, C, ldc, tm, ids, X, s);
  else if (cmode == 1)
    launch_dcb_t<KS, 1>(rf, L, C, ldc, tm, ids, X, s);
  else
    launch_dcb_t<KS, 2>(rf, L, C, ldc, tm, ids, X, s);
}

// Leading dimensions below 2^31 elements keep row x row-bytes products in
// 32-bit operands (the kernel's row addressing).
constexpr int64_t kMaxLd = int64_t{1} << 31;
bool table_ok(const void *T, int64_t ld) {
  return !T || (aligned16(T) && ld % 8 == 0 && ld < kMaxLd);
}

}  // namespace

bool decompress_mfma_ok(const PackLayout &L, void *X, int64_t ldx, const IdArgs &ids) {
  return L.mfma && L.d % kDCols == 0 && aligned16(X) && ldx % 8 == 0 && ldx < kMaxLd &&
         table_ok(ids.E, ids.lde) && table_ok(ids.P, ids.ldp);
}

hipError_t launch_decompress_mfma(const PackLayout &L, const void *packed, const void *C,
                                  int64_t N, int64_t ldc, const IdArgs &ids, void *X,
                                  int64_t ldx, hipStream_t s) {
  return launch_decompress_mfma_segs(L, packed, C, N, ldc, ids, one_seg(X, L.d, ldx), s);
}

hipError_t launch_decompress_mfma_segs(const PackLayout &L, const void *packed, const void *C,
                                       int64_t N, int64_t ldc, const IdArgs &ids,
                                       const ColSegs &X, hipStream_t s) {
  for (int i = 0; i < X.n; ++i)
    if (X.ld[i] % 8 != 0 || X.ld[i] >= kMaxLd) return hipErrorNotSupported;
  if (!table_ok(ids.E, ids.lde) || !table_ok(ids.P, ids.ldp)) return hipErrorNotSupported;
  const bf16_t *rf =
      reinterpret_cast<const bf16_t *>(static_cast<const char *>(packed) + L.off_rfrag);
  // how the coefficient rows may be read: 16-byte chunks, 4-byte pairs, or bf16 by bf16
  const uintptr_t ca = reinterpret_cast<uintptr_t>(C);
  const int cmode = (ca & 15) == 0 && ldc % 8 == 0 && L.k % 8 == 0   ? 0
                    : (ca & 3) == 0 && ldc % 2 == 0 && L.k % 2 == 0 ? 1
                                                                    : 2;
  DTiling tm{static_cast<int>(N), 0, 0};
  // position-major order for the default positions of [batch, seq] rows; a
  // short last sequence is allowed while the rows it lacks (read, not
  // stored) are at most an eighth of a sequence
  if (ids.P && !ids.pos && ids.seq_len % 16 == 0 && N >= ids.seq_len &&
      (ceil_div(N, ids.seq_len) * ids.seq_len - N) * 8 <= ids.seq_len &&
      ceil_div(N, ids.seq_len) * ids.seq_len <= INT32_MAX) {
    tm.seq = static_cast<int>(ids.seq_len);
    tm.batch = static_cast<int>(ceil_div(N, ids.seq_len));
  }
  switch (L.ks) {
    case 1: launch_dcb_ks<1>(rf, L, C, ldc, cmode, tm, ids, X, s); break;
    case 2: launch_dcb_ks<2>(rf, L, C, ldc, cmode, tm, ids, X, s); break;
    case 3: launch_dcb_ks<3>(rf, L, C, ldc, cmode, tm, ids, X, s); break;
    case 4: launch_dcb_ks<4>(rf, L, C, ldc, cmode, tm, ids, X, s); break;
    default: return hipErrorNotSupported;
  }
  return hipGetLastError();
}

}  // namespace sn
