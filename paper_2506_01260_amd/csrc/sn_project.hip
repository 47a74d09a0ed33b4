// Weight confinement W <- U (U^T W) on the gfx950 matrix cores.
#include "sn_mfma_common.h"

namespace sn {

namespace {

constexpr int kWaves = 4;  // waves per workgroup
constexpr int kBlock = 64 * kWaves;

}  // namespace

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
//
// When m is a multiple of 256 and k <= 64, pass 3 is the decompress kernel
// instead: W = U T_hi + U T_lo = [U | U] [T_hi ; T_lo] is a decompress of the
// d x 2k "coefficients" [U | U] (a section of the packed basis) against the
// m x 2k "basis" [T_hi | T_lo]^T, which pass 2 then writes in the decompress
// operand layout (rfrag).  That kernel keeps its 256-column slice of the
// basis in LDS and writes whole 256-byte row pieces.

namespace {

constexpr int kProjCols = 64;  // columns per workgroup in pass 3
constexpr int kPadCols = 128;  // m is padded to a multiple of the widest pass-1 slab

struct ProjPlan {
  int64_t m_pad;      // m rounded up to kProjCols
  int kp;             // 16 * kt: fp32 row length of Tp
  int kp32;           // 32 * ks: bf16 row length of Th / Tl
  int ks2;            // ceil(2k / 32): k-steps of [T_hi | T_lo]
  int dsplit;         // row splits in pass 1
  int64_t rows_per_split;
  size_t off_tp, off_th, off_tl, off_tr, total;
};

// Pass 1 splits the rows of W into dsplit ranges when there are too few
// column slabs to fill the chip; it picks the split that minimises
// (rounds of workgroups) x (rows per workgroup + a fixed cost of 256 rows:
// filling the load ring, the cross-wave reduction, the T writes) for `slots`
// resident workgroups (slots <= 0: the largest split, for the workspace
// bound).  Without the fixed cost, wide matrices were cut into many
// workgroups of a few row steps each.
ProjPlan proj_plan(int64_t k, int kt, int ks, int64_t m, int64_t d, int64_t slots) {
  ProjPlan P;
  P.m_pad = ceil_div(m, kPadCols) * kPadCols;
  P.kp = 16 * kt;
  P.kp32 = 32 * ks;
  P.ks2 = static_cast<int>(ceil_div(2 * k, 32));
  const int64_t slabs = ceil_div(m, 16 * (kt <= 4 ? 8 : 4));  // pass-1 workgroups per split
  int64_t max_ds = d / 128;  // >= 32 rows per wave
  if (max_ds > 8) max_ds = 8;
  // wide matrices (several weights side by side) fill the chip with few splits
  const int64_t by_cols = ceil_div(1024, slabs);
  if (max_ds > by_cols) max_ds = by_cols;
  if (max_ds < 1) max_ds = 1;
  int64_t best = max_ds, best_cost = -1;
  if (slots > 0) {
    for (int64_t ds = 1; ds <= max_ds; ++ds) {
      const int64_t rows = ceil_div(ceil_div(d, ds), 128) * 128;
      const int64_t cost = ceil_div(slabs * ceil_div(d, rows), slots) * (rows + 256);
      if (best_cost < 0 || cost < best_cost) {
        best = ds;
        best_cost = cost;
      }
    }
  }
  P.rows_per_split = ceil_div(ceil_div(d, best), 128) * 128;
  P.dsplit = static_cast<int>(ceil_div(d, P.rows_per_split));
  size_t off = 0;
  P.off_tp = off;
  off = align256(off + static_cast<size_t>(P.dsplit) * P.m_pad * P.kp * sizeof(float));
  P.off_th = off;
  off = align256(off + static_cast<size_t>(P.m_pad) * P.kp32 * 2);
  P.off_tl = off;
  off = align256(off + static_cast<size_t>(P.m_pad) * P.kp32 * 2);
  P.off_tr = off;  // [T_hi | T_lo] in the rfrag layout: m_pad x 32 ks2 bf16
  off = align256(off + static_cast<size_t>(P.m_pad) * 32 * P.ks2 * 2);
  P.total = off;
  return P;
}

// Columns per lane in pass 1: 8 (16-byte row loads) while the accumulators
// fit (KT <= 4), else 4 (8-byte loads).  A wave covers 16 * CW columns.
template <int KT>
constexpr int p1_cw() { return KT <= 4 ? 8 : 4; }

template <int CW> struct P1Vec;
template <> struct P1Vec<8> { typedef u32x4 T; };
template <> struct P1Vec<4> { typedef u32x2 T; };

// CLAMP: rows at or past nrows read row nrows - 1 instead (the caller's
// operand is zero there), for a reduction length that is not a multiple of
// the split size (the subspace update's contraction over tokens).
// Row steps in flight per wave: the weight projection at k <= 48 runs two
// waves per SIMD with a 2-deep ring (same bytes in flight per CU, twice the
// waves to issue them); otherwise one wave per SIMD with a 4-deep ring.
template <int KT, bool CLAMP>
constexpr bool p1_two_waves() { return !CLAMP && KT <= 3; }

template <int KT, bool CLAMP = false, int CW = p1_cw<KT>()>
__global__ __launch_bounds__(kBlock, (p1_two_waves<KT, CLAMP>() ? 2 : 1)) void project_pass1_kernel(
    const bf16_t *__restrict__ kfrag, int64_t d, ColSegs ws, int64_t rows_per_split,
    int64_t m_pad, float *__restrict__ Tp, int64_t nrows = 0) {
  constexpr int W32 = CW / 2;  // 32-bit words per lane and row
  typedef typename P1Vec<CW>::T vec;
  __shared__ f32x4 red[KT][CW][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 4, n = lane & 15;
  const int64_t cb = static_cast<int64_t>(blockIdx.x) * (16 * CW);
  // CLAMP (the token contraction) takes the splits last-first: the rows the
  // preceding pass read last are the likeliest still to be cached
  const int split = CLAMP ? static_cast<int>(gridDim.y - 1 - blockIdx.y) : blockIdx.y;
  // the column segment holding this block (blocks never straddle two)
  int sg = 0;
  while (sg + 1 < ws.n && cb >= ws.c0[sg + 1]) ++sg;
  const bf16_t *__restrict__ W = static_cast<const bf16_t *>(ws.base[sg]);
  const int64_t ldw = ws.ld[sg];
  const int64_t col = cb + CW * n;           // global column (T's layout)
  const int64_t lcol = col - ws.c0[sg];      // column within the segment
  const bool cvalid = col < ws.c0[sg + 1];   // widths % 8 == 0: all CW columns are valid

  const int steps = static_cast<int>(rows_per_split / 32);
  const int sb = static_cast<int>(split * (rows_per_split / 32));
  const int send = static_cast<int>(d / 32);
  const int s0 = sb + steps * wave / kWaves;
  int s1 = sb + steps * (wave + 1) / kWaves;
  if (s1 > send) s1 = send;

  f32x4 acc[KT][CW];
#pragma unroll
  for (int t = 0; t < KT; ++t)
#pragma unroll
    for (int q = 0; q < CW; ++q) acc[t][q] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Lanes past column m read column 0 instead (any finite values): every
  // load is unconditional and their columns are never stored.
  const bf16_t *wcol = W + (cvalid ? lcol : 0);
  const bf16_t *ufrag = kfrag + lane * 8;
  // rows 32 s + 8 g + e of the lane's CW columns, and the step's U fragments
  auto load = [&](int s, vec (&v)[8], u32x4 (&a)[KT]) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      int64_t row = 32 * static_cast<int64_t>(s) + 8 * g + e;
      if constexpr (CLAMP) row = row < nrows ? row : nrows - 1;
      v[e] = *reinterpret_cast<const vec *>(wcol + row * ldw);
    }
#pragma unroll
    for (int t = 0; t < KT; ++t) a[t] = ld16(ufrag + (static_cast<int64_t>(s) * KT + t) * 512);
  };
  auto word = [](const vec &v, int w) -> uint32_t {
    if constexpr (CW == 8) return w == 0 ? v.x : w == 1 ? v.y : w == 2 ? v.z : v.w;
    else return w == 0 ? v.x : v.y;
  };
  auto step = [&](const vec (&v)[8], const u32x4 (&a)[KT]) {
    // 8 x CW block (rows e, columns q) -> CW B operands of 8 rows each
#pragma unroll
    for (int w = 0; w < W32; ++w) {
      u32x4 b0, b1;  // columns 2 w and 2 w + 1
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t lo = word(v[2 * i], w), hi = word(v[2 * i + 1], w);
        b0[i] = __builtin_amdgcn_perm(hi, lo, 0x05040100u);  // low halves
        b1[i] = __builtin_amdgcn_perm(hi, lo, 0x07060302u);  // high halves
      }
#pragma unroll
      for (int t = 0; t < KT; ++t) {
        acc[t][2 * w] = mfma(a[t], b0, acc[t][2 * w]);
        acc[t][2 * w + 1] = mfma(a[t], b1, acc[t][2 * w + 1]);
      }
    }
  };

  // PD-deep ring of row steps in flight (memory latency under load is long):
  // step s + PD is loaded as soon as step s has been consumed; past the end
  // the last step is reloaded.
  constexpr int PD = p1_two_waves<KT, CLAMP>() ? 2 : 4;
  if (s0 < s1) {
    vec v[PD][8];
    u32x4 a[PD][KT];
#pragma unroll
    for (int r = 0; r < PD; ++r) load(s0 + r < s1 ? s0 + r : s1 - 1, v[r], a[r]);
    int s = s0;
    for (; s + PD <= s1; s += PD) {  // whole groups: no guards in the loop body
#pragma unroll
      for (int r = 0; r < PD; ++r) {
        step(v[r], a[r]);
        const int sn = s + r + PD;
        load(sn < s1 ? sn : s1 - 1, v[r], a[r]);
        __builtin_amdgcn_sched_barrier(0);  // keep the refill here
      }
    }
#pragma unroll
    for (int r = 0; r < PD; ++r)
      if (s + r < s1) step(v[r], a[r]);
  }

  // fixed-order reduction: acc0 + (acc1 + (acc2 + acc3))
  for (int w = kWaves - 1; w >= 1; --w) {
    if (wave == w) {
#pragma unroll
      for (int t = 0; t < KT; ++t)
#pragma unroll
        for (int q = 0; q < CW; ++q) {
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
      for (int q = 0; q < CW; ++q) {
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

// pass 2 for the decompress-form pass 3: one thread per (column c, j) with
// j < 16 ks2; for j < k it writes T_hi[j, c] and T_lo[j, c] (k-indices j and
// k + j of [T_hi | T_lo]), past k two of the zero pad entries.
__global__ __launch_bounds__(256) void project_pass2_rfrag_kernel(
    const float *__restrict__ Tp, int dsplit, int64_t m, int64_t m_pad, int kp, int64_t k,
    int ks2, bf16_t *__restrict__ tr) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int half = 16 * ks2;
  if (idx >= m * half) return;
  const int64_t c = idx / half;
  const int j = static_cast<int>(idx - c * half);
  bf16_t v0 = bf16_t(0), v1 = bf16_t(0);
  int j0, j1;
  if (j < k) {
    // every split's value first (independent loads in flight together), then
    // the fixed-order compensated sum; dsplit <= 8
    float t[8];
#pragma unroll
    for (int sp = 0; sp < 8; ++sp)
      t[sp] = sp < dsplit ? Tp[((sp < dsplit ? sp : 0) * m_pad + c) * kp + j] : 0.0f;
    Dot2 acc;
#pragma unroll
    for (int sp = 0; sp < 8; ++sp)
      if (sp < dsplit) acc.add(t[sp]);
    const float v = acc.value();
    v0 = from_f32<bf16_t>(v);
    v1 = from_f32<bf16_t>(v - to_f32(v0));
    j0 = j;
    j1 = static_cast<int>(k) + j;
  } else {
    j0 = static_cast<int>(2 * k + 2 * (j - k));
    j1 = j0 + 1;
  }
  // rfrag slot of basis row c, k-index j2 (the packed-basis rfrag layout)
  const int64_t p = c / 32;
  const int rr = static_cast<int>(c - 32 * p);
  const int h = (rr >> 2) & 1, mm = 4 * (rr >> 3) + (rr & 3);
  auto put = [&](int j2, bf16_t x) {
    const int q = j2 >> 5, g = (j2 & 31) >> 3, e = j2 & 7;
    tr[(((p * 2 + h) * ks2 + q) * 64 + 16 * g + mm) * 8 + e] = x;
  };
  put(j0, v0);
  put(j1, v1);
}

template <int KS>
__global__ __launch_bounds__(kBlock) void project_pass3_kernel(
    const bf16_t *__restrict__ rfrag, int64_t d, const bf16_t *__restrict__ Th,
    const bf16_t *__restrict__ Tl, bf16_t *__restrict__ W, int64_t m, int64_t ldw,
    int64_t rows_per_block) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
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

  // U fragments of row group p (loaded one group ahead; past the end the
  // last group is reloaded)
  auto load_u = [&](int p, u32x4 (&b)[2][KS]) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int q = 0; q < KS; ++q)
        b[h][q] = ld16(ufrag + ((static_cast<int64_t>(p) * 2 + h) * KS + q) * 512);
  };
  auto group = [&](int p, const u32x4 (&b)[2][KS]) {
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
  };
  if (p0 < p1) {
    u32x4 b0[2][KS], b1[2][KS];
    load_u(p0, b0);
    int p = p0;
    for (; p + 2 <= p1; p += 2) {
      load_u(p + 1, b1);
      group(p, b0);
      load_u(p + 2 < p1 ? p + 2 : p1 - 1, b0);
      group(p + 1, b1);
    }
    if (p < p1) group(p, b0);
  }
}

template <int KT>
void launch_p1(const ProjPlan &P, const bf16_t *kf, int64_t d, const ColSegs &W, int64_t m,
               float *Tp, hipStream_t s) {
  dim3 grid(static_cast<unsigned>(ceil_div(m, 16 * p1_cw<KT>())), static_cast<unsigned>(P.dsplit));
  project_pass1_kernel<KT><<<grid, kBlock, 0, s>>>(kf, d, W, P.rows_per_split, P.m_pad, Tp);
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

template <int KT>
int64_t slots_kt() {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &per_cu, reinterpret_cast<const void *>(project_pass1_kernel<KT>), kBlock, 0) !=
          hipSuccess)
    return 256;
  return static_cast<int64_t>(cus) * (per_cu > 0 ? per_cu : 1);
}

// resident pass-1 workgroups on the current device
int64_t pass1_slots(int kt) {
  switch (kt) {
    case 1: return slots_kt<1>();
    case 2: return slots_kt<2>();
    case 3: return slots_kt<3>();
    case 4: return slots_kt<4>();
    case 5: return slots_kt<5>();
    case 6: return slots_kt<6>();
    case 7: return slots_kt<7>();
    default: return slots_kt<8>();
  }
}

}  // namespace

// Subspace update, contraction over tokens: Tp[split][i][j] = sum over the
// split's rows n of F[n, j] G[n, i], F the (npad x 16 ktb) operand in the kfrag
// layout (zero past N), G the N x d gradient; the pass-1 kernel with the
// roles d -> tokens, W -> G, U -> F.
// 16-byte row pieces (8 columns per lane) up to 5 column tiles: the
// accumulators then live in the AGPRs
template <int KT>
constexpr int tok_cw() { return KT <= 5 ? 8 : 4; }

template <int KT>
void launch_p1_tokens(const bf16_t *frag, int64_t npad, const bf16_t *G, int64_t N, int64_t ldg,
                      int64_t d, int64_t rows, int ds, int64_t m_pad, float *Tp, hipStream_t s) {
  constexpr int CW = tok_cw<KT>();
  dim3 grid(static_cast<unsigned>(ceil_div(d, 16 * CW)), static_cast<unsigned>(ds));
  project_pass1_kernel<KT, true, CW><<<grid, kBlock, 0, s>>>(frag, npad, one_seg(G, d, ldg),
                                                              rows, m_pad, Tp, N);
}

hipError_t launch_grass_tokens_mfma(const void *frag, int ktb, int64_t npad, const void *G,
                                    int64_t N, int64_t ldg, int64_t d, int64_t rows, int ds,
                                    int64_t m_pad, float *Tp, hipStream_t s) {
  const bf16_t *f = static_cast<const bf16_t *>(frag);
  const bf16_t *g = static_cast<const bf16_t *>(G);
  switch (ktb) {
    case 1: launch_p1_tokens<1>(f, npad, g, N, ldg, d, rows, ds, m_pad, Tp, s); break;
    case 2: launch_p1_tokens<2>(f, npad, g, N, ldg, d, rows, ds, m_pad, Tp, s); break;
    case 3: launch_p1_tokens<3>(f, npad, g, N, ldg, d, rows, ds, m_pad, Tp, s); break;
    case 4: launch_p1_tokens<4>(f, npad, g, N, ldg, d, rows, ds, m_pad, Tp, s); break;
    case 5: launch_p1_tokens<5>(f, npad, g, N, ldg, d, rows, ds, m_pad, Tp, s); break;
    case 6: launch_p1_tokens<6>(f, npad, g, N, ldg, d, rows, ds, m_pad, Tp, s); break;
    case 7: launch_p1_tokens<7>(f, npad, g, N, ldg, d, rows, ds, m_pad, Tp, s); break;
    case 8: launch_p1_tokens<8>(f, npad, g, N, ldg, d, rows, ds, m_pad, Tp, s); break;
    default: return hipErrorNotSupported;
  }
  return hipGetLastError();
}

size_t project_workspace_mfma(int64_t d, int64_t k, int64_t m) {
  const int kt = static_cast<int>(ceil_div(k, 16)), ks = static_cast<int>(ceil_div(k, 32));
  return proj_plan(k, kt, ks, m, d, 0).total;  // the largest split bounds every plan
}

bool project_mfma_ok(const PackLayout &L, const void *W, int64_t m, int64_t ldw) {
  return L.mfma && aligned16(W) && ldw % 8 == 0 && m % 8 == 0 && L.d % 128 == 0;
}

hipError_t launch_project_mfma(const PackLayout &L, const void *packed, void *Wv, int64_t m,
                               int64_t ldw, void *ws, hipStream_t s) {
  return launch_project_mfma_segs(L, packed, one_seg(Wv, m, ldw), ws, s);
}

hipError_t launch_project_mfma_segs(const PackLayout &L, const void *packed, const ColSegs &W,
                                   void *ws, hipStream_t s) {
  const int64_t m = W.c0[W.n];
  const ProjPlan P = proj_plan(L.k, L.kt, L.ks, m, L.d, pass1_slots(L.kt));
  const char *base = static_cast<const char *>(packed);
  const bf16_t *kf = reinterpret_cast<const bf16_t *>(base + L.off_kfrag);
  const bf16_t *rf = reinterpret_cast<const bf16_t *>(base + L.off_rfrag);
  char *w = static_cast<char *>(ws);
  float *Tp = reinterpret_cast<float *>(w + P.off_tp);
  bf16_t *Th = reinterpret_cast<bf16_t *>(w + P.off_th);
  bf16_t *Tl = reinterpret_cast<bf16_t *>(w + P.off_tl);
  switch (L.kt) {
    case 1: launch_p1<1>(P, kf, L.d, W, m, Tp, s); break;
    case 2: launch_p1<2>(P, kf, L.d, W, m, Tp, s); break;
    case 3: launch_p1<3>(P, kf, L.d, W, m, Tp, s); break;
    case 4: launch_p1<4>(P, kf, L.d, W, m, Tp, s); break;
    case 5: launch_p1<5>(P, kf, L.d, W, m, Tp, s); break;
    case 6: launch_p1<6>(P, kf, L.d, W, m, Tp, s); break;
    case 7: launch_p1<7>(P, kf, L.d, W, m, Tp, s); break;
    case 8: launch_p1<8>(P, kf, L.d, W, m, Tp, s); break;
    default: return hipErrorNotSupported;
  }
  if (L.ks2 > 0 && m % 256 == 0) {
    // pass 3 as a decompress of [U | U] against [T_hi | T_lo]
    bf16_t *tr = reinterpret_cast<bf16_t *>(w + P.off_tr);
    const bf16_t *uu = reinterpret_cast<const bf16_t *>(base + L.off_uu);
    const int64_t n2 = m * 16 * P.ks2;
    project_pass2_rfrag_kernel<<<dim3(static_cast<unsigned>(ceil_div(n2, 256))), 256, 0, s>>>(
        Tp, P.dsplit, m, P.m_pad, P.kp, L.k, P.ks2, tr);
    PackLayout V;  // the m x 2k "basis" [T_hi | T_lo]^T, rfrag section only
    V.d = m;
    V.k = 2 * L.k;
    V.dt = 1;
    V.mfma = true;
    V.kt = static_cast<int>(ceil_div(V.k, 16));
    V.ks = P.ks2;
    V.off_rfrag = P.off_tr;
    IdArgs none{};
    const hipError_t e = launch_decompress_mfma_segs(V, ws, uu, L.d, 32 * P.ks2, none, W, s);
    return e != hipSuccess ? e : hipGetLastError();
  }
  if (W.n != 1) return hipErrorNotSupported;  // the segmented form needs widths % 256 == 0
  const int64_t n2 = P.m_pad * P.kp32;
  project_pass2_kernel<<<dim3(static_cast<unsigned>(ceil_div(n2, 256))), 256, 0, s>>>(
      Tp, P.dsplit, m, P.m_pad, P.kp, P.kp32, Th, Tl);
  bf16_t *Wp = static_cast<bf16_t *>(W.base[0]);
  const int64_t ldw = W.ld[0];
  switch (L.ks) {
    case 1: launch_p3<1>(P, rf, L.d, Th, Tl, Wp, m, ldw, s); break;
    case 2: launch_p3<2>(P, rf, L.d, Th, Tl, Wp, m, ldw, s); break;
    case 3: launch_p3<3>(P, rf, L.d, Th, Tl, Wp, m, ldw, s); break;
    case 4: launch_p3<4>(P, rf, L.d, Th, Tl, Wp, m, ldw, s); break;
    default: return hipErrorNotSupported;
  }
  return hipGetLastError();
}

}  // namespace sn
