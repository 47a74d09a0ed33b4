// The trainable low-rank token table of Sec. 4.3.1, kept as coefficients:
// T_S = C_S U^T (vocab x k coefficients), so its rows stay in S whatever
// C_S's optimizer does.  TE = T_fixed[t] + T_S[t].
//
// forward   X0[i] = P[pos_i] + T_fixed[tok_i] + C_S[tok_i] U^T: the C_S rows
//           of the batch are gathered into a coefficient buffer and the
//           decompress kernel does the rest (it is exactly Sec. 4.3.1's
//           recovery with C = C_S[tok]).
// backward  gC_S[v] += sum over i with tok_i = v of dX0[i] U: the gradient
//           coefficients dX0 U in fp32 (the compress kernel's fp32-row
//           epilogue), then a deterministic segmented sum by token id: a
//           stable counting sort of the token indices (per-block id
//           histograms, per-id prefixes over the blocks, one scan over the
//           vocabulary, and a bitonic sort of each block's (id, index) keys
//           in LDS for the ranks within a block), per-chunk sums of at most
//           64 rows of a segment, and per-segment sums of its chunks, every
//           sum in a fixed order in float64.
#include "sn_device.h"
#include "sn_internal.h"

namespace sn {

namespace {

constexpr int kSortThreads = 1024;

__device__ __forceinline__ int64_t ceil_div_dev(int64_t a, int64_t b) { return (a + b - 1) / b; }
constexpr int kChunk = 64;  // rows per chunk of a segment

struct EmbedPlan {
  int64_t kp = 0, maxseg = 0, maxchunk = 0, nblk = 0, ntile = 0;
  size_t off_lz = 0, off_lch = 0, off_tiles = 0, off_count = 0;
  size_t off_c = 0, off_cnt = 0, off_cur = 0, off_order = 0, off_segid = 0, off_segoff = 0,
         off_segch = 0, off_cbeg = 0, off_cend = 0, off_meta = 0, off_part = 0, total = 0;
};

EmbedPlan embed_plan(int64_t k, int dt, int64_t N, int64_t vocab, bool backward) {
  EmbedPlan P;
  P.kp = 16 * ceil_div(k, 16);
  size_t off = 0;
  P.off_c = off;
  // forward: the gathered coefficients (N x k, dt); backward: fp32 rows of kp
  const size_t cbytes = backward ? static_cast<size_t>(N) * P.kp * 4
                                 : static_cast<size_t>(N) * k * (dt == 0 ? 4 : 2);
  off = align256(off + cbytes);
  if (!backward) {
    P.total = off;
    return P;
  }
  P.maxseg = N < vocab ? N : vocab;
  P.maxchunk = ceil_div(N, kChunk) + P.maxseg;
  P.nblk = ceil_div(N, kSortThreads);
  auto ints = [&](size_t &o, int64_t n) {
    o = off;
    off = align256(off + static_cast<size_t>(n) * 4);
  };
  ints(P.off_cnt, P.nblk * vocab);  // per-block id counts, then their prefixes over blocks
  ints(P.off_cur, vocab);           // per-id totals, then the ids' first slots
  P.ntile = ceil_div(vocab, kSortThreads);
  ints(P.off_count, vocab);         // per-id token counts
  ints(P.off_lz, vocab);            // per id: segments and chunks before it in its tile
  ints(P.off_lch, vocab);
  ints(P.off_tiles, 6 * P.ntile);   // per tile: tokens, segments, chunks; then their offsets
  ints(P.off_order, N);
  ints(P.off_segid, P.maxseg);
  ints(P.off_segoff, P.maxseg + 1);
  ints(P.off_segch, P.maxseg + 1);
  ints(P.off_cbeg, P.maxchunk);
  ints(P.off_cend, P.maxchunk);
  ints(P.off_meta, 4);
  P.off_part = off;
  off = align256(off + static_cast<size_t>(P.maxchunk) * P.kp * 8);
  P.total = off;
  return P;
}

// C[i, :] = C_S[tok_i, :] (ids clamped into [0, vocab), bit 0 of *err_flag)
template <typename T>
__global__ __launch_bounds__(256) void gather_rows_kernel(const T *__restrict__ CS, int64_t ldcs,
                                                          const int32_t *__restrict__ tok,
                                                          int64_t vocab, int64_t N, int64_t k,
                                                          T *__restrict__ C,
                                                          int32_t *err_flag) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= N * k) return;
  const int64_t i = idx / k, j = idx - (idx / k) * k;
  int64_t v = tok[i];
  if (v < 0 || v >= vocab) {
    if (err_flag && j == 0) atomicOr(err_flag, 1);
    v = v < 0 ? 0 : vocab - 1;
  }
  C[idx] = CS[v * ldcs + j];
}

// Exclusive scan of one int per thread over the 1024 threads (Hillis-Steele
// in LDS); *total receives the sum.
__device__ int block_excl_scan(int v, int *buf, int *total) {
  const int t = threadIdx.x;
  buf[t] = v;
  __syncthreads();
  for (int off = 1; off < kSortThreads; off <<= 1) {
    const int add = t >= off ? buf[t - off] : 0;
    __syncthreads();
    buf[t] += add;
    __syncthreads();
  }
  const int incl = buf[t];
  *total = buf[kSortThreads - 1];
  __syncthreads();
  return incl - v;
}

__device__ __forceinline__ int clamp_tok(const int32_t *tok, int64_t i, int64_t vocab,
                                         int32_t *err_flag) {
  int64_t v = tok[i];
  if (v < 0 || v >= vocab) {
    if (err_flag) atomicOr(err_flag, 1);
    v = v < 0 ? 0 : vocab - 1;
  }
  return static_cast<int>(v);
}

// cnt[b][v] = number of tokens of block b (1024 tokens each) with id v; the
// block clears its own row first (the barrier orders the clearing stores
// before the block's increments)
__global__ __launch_bounds__(kSortThreads) void hist_kernel(const int32_t *__restrict__ tok,
                                                            int64_t N, int64_t vocab,
                                                            int32_t *err_flag,
                                                            int32_t *__restrict__ cnt) {
  int32_t *row = cnt + static_cast<int64_t>(blockIdx.x) * vocab;
  for (int64_t v = threadIdx.x; v < vocab; v += kSortThreads) row[v] = 0;
  __syncthreads();
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kSortThreads + threadIdx.x;
  if (i < N) atomicAdd(&row[clamp_tok(tok, i, vocab, err_flag)], 1);
}

// per id v: cnt[b][v] <- tokens of id v in the blocks before b; tot[v] <- all of them
__global__ __launch_bounds__(256) void block_prefix_kernel(int32_t *__restrict__ cnt,
                                                           int64_t nblk, int64_t vocab,
                                                           int32_t *__restrict__ tot,
                                                           int32_t *__restrict__ count) {
  const int64_t v = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (v >= vocab) return;
  int run = 0;
  for (int64_t b = 0; b < nblk; ++b) {
    const int c = cnt[b * vocab + v];
    cnt[b * vocab + v] = run;
    run += c;
  }
  tot[v] = run;
  count[v] = run;
}

// Scan over the vocabulary in three kernels.  Tile pass: per 1024-id tile,
// exclusive prefixes within the tile of the ids' token counts, of the ids
// that occur (segments) and of their chunks (at most kChunk rows each), and
// the tile's three totals.
__global__ __launch_bounds__(kSortThreads) void tile_scan_kernel(
    int64_t vocab, int32_t *__restrict__ tot, int32_t *__restrict__ lz,
    int32_t *__restrict__ lch, int32_t *__restrict__ tiles, int64_t ntile) {
  __shared__ int buf[kSortThreads];
  const int64_t v = static_cast<int64_t>(blockIdx.x) * kSortThreads + threadIdx.x;
  const int c = v < vocab ? tot[v] : 0;
  int sc, sz, sch;
  const int ec = block_excl_scan(c, buf, &sc);
  const int ez = block_excl_scan(c > 0, buf, &sz);
  const int ech = block_excl_scan((c + kChunk - 1) / kChunk, buf, &sch);
  if (v < vocab) {
    tot[v] = ec;
    lz[v] = ez;
    lch[v] = ech;
  }
  if (threadIdx.x == 0) {
    tiles[blockIdx.x] = sc;
    tiles[ntile + blockIdx.x] = sz;
    tiles[2 * ntile + blockIdx.x] = sch;
  }
}

// One workgroup: exclusive prefixes of the tiles' totals (into tiles[3 ntile
// ..]), the segment and chunk counts, and the end markers of both tables.
__global__ __launch_bounds__(kSortThreads) void tiles_scan_kernel(
    int64_t N, int32_t *__restrict__ tiles, int64_t ntile, int32_t *__restrict__ seg_off,
    int32_t *__restrict__ seg_ch, int32_t *__restrict__ meta) {
  __shared__ int buf[kSortThreads];
  const int64_t per = ceil_div_dev(ntile, kSortThreads);
  const int64_t t0 = threadIdx.x * per < ntile ? threadIdx.x * per : ntile;
  const int64_t t1 = t0 + per < ntile ? t0 + per : ntile;
  for (int a = 0; a < 3; ++a) {
    int sum = 0;
    for (int64_t i = t0; i < t1; ++i) sum += tiles[a * ntile + i];
    int total;
    int run = block_excl_scan(sum, buf, &total);
    for (int64_t i = t0; i < t1; ++i) {
      const int c = tiles[a * ntile + i];
      tiles[(3 + a) * ntile + i] = run;
      run += c;
    }
    if (threadIdx.x == 0 && a == 1) meta[0] = total;
    if (threadIdx.x == 0 && a == 2) meta[1] = total;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    seg_off[meta[0]] = static_cast<int>(N);
    seg_ch[meta[0]] = meta[1];
  }
}

// Per id: its first slot, and for an id that occurs its segment entry and
// chunk table entries.
__global__ __launch_bounds__(kSortThreads) void tile_write_kernel(
    int64_t vocab, const int32_t *__restrict__ cnt_last, int64_t nblk, int32_t *__restrict__ tot,
    const int32_t *__restrict__ lz, const int32_t *__restrict__ lch,
    const int32_t *__restrict__ tiles, int64_t ntile, int32_t *__restrict__ seg_id,
    int32_t *__restrict__ seg_off, int32_t *__restrict__ seg_ch, int32_t *__restrict__ cbeg,
    int32_t *__restrict__ cend, const int32_t *__restrict__ count) {
  const int64_t tile = blockIdx.x;
  const int64_t v = tile * kSortThreads + threadIdx.x;
  if (v >= vocab) return;
  const int first = tiles[3 * ntile + tile] + tot[v];
  tot[v] = first;
  const int c = count[v];
  if (c == 0) return;
  const int sgi = tiles[4 * ntile + tile] + lz[v];
  int q = tiles[5 * ntile + tile] + lch[v];
  seg_id[sgi] = static_cast<int>(v);
  seg_off[sgi] = first;
  seg_ch[sgi] = q;
  for (int b = 0; b < c; b += kChunk, ++q) {
    cbeg[q] = first + b;
    cend[q] = first + (b + kChunk < c ? b + kChunk : c);
  }
  (void)cnt_last;
  (void)nblk;
}

// Block b's tokens in sorted order: keys (id << 10 | local index) sorted in
// LDS (bitonic), a token's rank among the block's tokens of its id is its
// sorted position minus the first position of its id (a max scan of the run
// heads), and its slot is first[id] + (id's tokens in earlier blocks) + rank.
// Ids must be below 2^21.
__global__ __launch_bounds__(kSortThreads) void place_kernel(
    const int32_t *__restrict__ tok, int64_t N, int64_t vocab, const int32_t *__restrict__ cnt,
    const int32_t *__restrict__ first, int32_t *__restrict__ order) {
  __shared__ uint32_t key[kSortThreads];
  __shared__ int hs[kSortThreads];
  const int t = threadIdx.x;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kSortThreads;
  const int64_t i = base + t;
  key[t] = i < N ? (static_cast<uint32_t>(clamp_tok(tok, i, vocab, nullptr)) << 10) |
                       static_cast<uint32_t>(t)
                 : 0xFFFFFFFFu;
  __syncthreads();
  for (int kk = 2; kk <= kSortThreads; kk <<= 1) {
    for (int j = kk >> 1; j > 0; j >>= 1) {
      const int p = t ^ j;
      if (p > t) {
        const uint32_t a = key[t], b = key[p];
        if ((a > b) == ((t & kk) == 0)) {
          key[t] = b;
          key[p] = a;
        }
      }
      __syncthreads();
    }
  }
  const uint32_t me = key[t];
  const bool head = t == 0 || (key[t - 1] >> 10) != (me >> 10);
  hs[t] = head ? t : 0;
  __syncthreads();
  for (int off = 1; off < kSortThreads; off <<= 1) {  // inclusive max scan
    const int o = t >= off ? hs[t - off] : 0;
    __syncthreads();
    hs[t] = hs[t] > o ? hs[t] : o;
    __syncthreads();
  }
  if (me != 0xFFFFFFFFu) {
    const int64_t id = me >> 10;
    const int rank = t - hs[t];
    const int64_t slot = first[id] + cnt[static_cast<int64_t>(blockIdx.x) * vocab + id] + rank;
    order[slot] = static_cast<int32_t>(base + (me & 1023u));
  }
}

// One wave per chunk: part[q][j] = sum over the chunk's rows (ascending
// token index) of c32[row][j], float64.  Lane r copies row r of the chunk
// into LDS (contiguous loads), then lane j adds column j down the rows.
__global__ __launch_bounds__(256) void chunk_sum_kernel(const float *__restrict__ c32, int64_t kp,
                                                        const int32_t *__restrict__ order,
                                                        const int32_t *__restrict__ cbeg,
                                                        const int32_t *__restrict__ cend,
                                                        const int32_t *__restrict__ meta,
                                                        double *__restrict__ part) {
  constexpr int JC = 64, LD = JC + 1;  // columns per pass, LDS row stride
  __shared__ float rows[4][kChunk * LD];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 4 + w;
  const bool live = q < meta[1];
  const int b = live ? cbeg[q] : 0, len = live ? cend[q] - b : 0;
  float *rw = rows[w];
  for (int64_t j0 = 0; j0 < kp; j0 += JC) {  // same trip count in every wave
    const int64_t jn = kp - j0 < JC ? kp - j0 : JC;
    if (lane < len) {
      const float *src = c32 + static_cast<int64_t>(order[b + lane]) * kp + j0;
      for (int64_t j = 0; j < jn; ++j) rw[lane * LD + j] = src[j];
    }
    __syncthreads();
    if (live && lane < jn) {
      double acc = 0.0;
      for (int r = 0; r < len; ++r) acc += static_cast<double>(rw[r * LD + lane]);
      part[q * kp + j0 + lane] = acc;
    }
    __syncthreads();
  }
}

// One wave per segment: gCS[v][j] += the segment's chunk sums, in order.
__global__ __launch_bounds__(256) void seg_sum_kernel(const double *__restrict__ part, int64_t kp,
                                                      int64_t k, const int32_t *__restrict__ seg_id,
                                                      const int32_t *__restrict__ seg_ch,
                                                      const int32_t *__restrict__ meta,
                                                      float *__restrict__ gCS, int64_t ldgc) {
  const int lane = threadIdx.x & 63;
  const int64_t s = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (s >= meta[0]) return;
  const int64_t v = seg_id[s];
  const int q0 = seg_ch[s], q1 = seg_ch[s + 1];
  for (int64_t j = lane; j < k; j += 64) {
    double acc = 0.0;
    for (int q = q0; q < q1; ++q) acc += part[static_cast<int64_t>(q) * kp + j];
    gCS[v * ldgc + j] += static_cast<float>(acc);
  }
}

}  // namespace

size_t embed_workspace_bytes(int64_t k, int dt, int64_t N, int64_t vocab) {
  const size_t f = embed_plan(k, dt, N, vocab, false).total;
  const size_t b = embed_plan(k, dt, N, vocab, true).total;
  return f > b ? f : b;
}

hipError_t launch_embed_forward(const PackLayout &L, const void *packed, const void *CS,
                                int64_t vocab, int64_t ldcs, const int32_t *tok,
                                const IdArgs &ids, int64_t N, void *X0, int64_t ldx, void *ws,
                                hipStream_t s) {
  const EmbedPlan P = embed_plan(L.k, L.dt, N, vocab, false);
  void *C = static_cast<char *>(ws) + P.off_c;
  const dim3 grid(static_cast<unsigned>(ceil_div(N * L.k, 256)));
  if (L.dt == 0)
    gather_rows_kernel<float><<<grid, 256, 0, s>>>(static_cast<const float *>(CS), ldcs, tok,
                                                   vocab, N, L.k, static_cast<float *>(C),
                                                   ids.err_flag);
  else
    gather_rows_kernel<bf16_t><<<grid, 256, 0, s>>>(static_cast<const bf16_t *>(CS), ldcs, tok,
                                                    vocab, N, L.k, static_cast<bf16_t *>(C),
                                                    ids.err_flag);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  if (decompress_mfma_ok(L, X0, ldx, ids))
    return launch_decompress_mfma(L, packed, C, N, L.k, ids, X0, ldx, s);
  return launch_decompress_generic(L, packed, C, N, L.k, ids, X0, ldx, s);
}

hipError_t launch_embed_backward(const PackLayout &L, const void *packed, const void *dX0,
                                 int64_t N, int64_t ldg, const int32_t *tok, int64_t vocab,
                                 float *gCS, int64_t ldgc, int32_t *err_flag, void *ws,
                                 hipStream_t s) {
  const EmbedPlan P = embed_plan(L.k, L.dt, N, vocab, true);
  char *w = static_cast<char *>(ws);
  float *c32 = reinterpret_cast<float *>(w + P.off_c);
  hipError_t e = stream_mfma_ok(L, dX0, ldg)
                     ? launch_table_project_mfma(L, packed, dX0, N, ldg, c32, P.kp, s)
                     : launch_table_project_generic(L, packed, dX0, N, ldg, c32, P.kp, s);
  if (e != hipSuccess) return e;
  auto I = [&](size_t off) { return reinterpret_cast<int32_t *>(w + off); };
  hist_kernel<<<dim3(static_cast<unsigned>(P.nblk)), kSortThreads, 0, s>>>(tok, N, vocab,
                                                                           err_flag, I(P.off_cnt));
  block_prefix_kernel<<<dim3(static_cast<unsigned>(ceil_div(vocab, 256))), 256, 0, s>>>(
      I(P.off_cnt), P.nblk, vocab, I(P.off_cur), I(P.off_count));
  tile_scan_kernel<<<dim3(static_cast<unsigned>(P.ntile)), kSortThreads, 0, s>>>(
      vocab, I(P.off_cur), I(P.off_lz), I(P.off_lch), I(P.off_tiles), P.ntile);
  tiles_scan_kernel<<<dim3(1), kSortThreads, 0, s>>>(N, I(P.off_tiles), P.ntile, I(P.off_segoff),
                                                      I(P.off_segch), I(P.off_meta));
  tile_write_kernel<<<dim3(static_cast<unsigned>(P.ntile)), kSortThreads, 0, s>>>(
      vocab, nullptr, 0, I(P.off_cur), I(P.off_lz), I(P.off_lch), I(P.off_tiles), P.ntile,
      I(P.off_segid), I(P.off_segoff), I(P.off_segch), I(P.off_cbeg), I(P.off_cend),
      I(P.off_count));
  place_kernel<<<dim3(static_cast<unsigned>(P.nblk)), kSortThreads, 0, s>>>(
      tok, N, vocab, I(P.off_cnt), I(P.off_cur), I(P.off_order));
  double *part = reinterpret_cast<double *>(w + P.off_part);
  chunk_sum_kernel<<<dim3(static_cast<unsigned>(ceil_div(P.maxchunk, 4))), 256, 0, s>>>(
      c32, P.kp, I(P.off_order), I(P.off_cbeg), I(P.off_cend), I(P.off_meta), part);
  seg_sum_kernel<<<dim3(static_cast<unsigned>(ceil_div(P.maxseg, 4))), 256, 0, s>>>(
      part, P.kp, L.k, I(P.off_segid), I(P.off_segch), I(P.off_meta), gCS, ldgc);
  return hipGetLastError();
}

}  // namespace sn
