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
//           epilogue), then a deterministic sum by token id in two kernels:
//           per block of 512 tokens, a bitonic sort of the (id, index) keys
//           and, per run of equal ids, the float64 sum of its rows in
//           ascending token order; per id, the sum of its runs over the
//           blocks in block order (float64), added to gC_S.
#include "sn_device.h"
#include "sn_internal.h"

namespace sn {

namespace {

constexpr int kBlk = 512;      // tokens per sort block (threads of block_runs_kernel)
constexpr int kBlkWaves = kBlk / 64;
constexpr int kIdRange = 64;   // ids per workgroup of id_merge_kernel

struct EmbedPlan {
  int64_t kp = 0, nblk = 0, nq = 0;
  size_t off_c = 0, off_rid = 0, off_first = 0, off_part = 0, total = 0;
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
  P.nblk = ceil_div(N, kBlk);
  P.nq = ceil_div(vocab, kIdRange);
  P.off_rid = off;  // per block: the ids of its runs, ascending
  off = align256(off + static_cast<size_t>(P.nblk) * kBlk * 4);
  P.off_first = off;  // per block: the first run of each range of kIdRange ids, then the runs
  off = align256(off + static_cast<size_t>(P.nblk) * (P.nq + 1) * 4);
  P.off_part = off;  // per block and run: the float64 sum of the run's rows
  off = align256(off + static_cast<size_t>(P.nblk) * kBlk * P.kp * 8);
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

// Exclusive count of the flags of the threads before this one in the block,
// and the block's total: ballots within each wave, the waves' counts through
// LDS (wtot holds kBlkWaves ints).
__device__ int block_excl_count(bool flag, int *wtot, int *total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const uint64_t m = __ballot(flag);
  if (lane == 0) wtot[w] = __popcll(m);
  __syncthreads();
  int before = __popcll(m & ((1ull << lane) - 1ull)), all = 0;
#pragma unroll
  for (int i = 0; i < kBlkWaves; ++i) {
    const int c = wtot[i];
    before += i < w ? c : 0;
    all += c;
  }
  *total = all;
  return before;
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

// Block b (tokens base .. base + 511): the keys (id << 9 | local index)
// sorted (bitonic), so each run of equal ids lists its tokens in
// ascending order.  rid[b][r] = the id of run r (ascending); first[b][q] =
// the first run with an id of at least q kIdRange (q = 0 .. nq, first[b][nq]
// = the runs); part[b][r][:] = the float64 sum of the run's c32 rows in
// order.  Wave w sums the sorted positions 64 w .. 64 w + 63 (lane = column,
// 64 columns per pass): a run that begins and ends inside the wave is written
// directly; a run that crosses waves leaves its first and middle pieces in
// LDS and the wave where it ends adds them in order.  Ids must be below 2^21.
__global__ __launch_bounds__(kBlk) void block_runs_kernel(
    const int32_t *__restrict__ tok, int64_t N, int64_t vocab, int32_t *err_flag,
    const float *__restrict__ c32, int kp, int64_t nq, int32_t *__restrict__ rid_out,
    int32_t *__restrict__ first, double *__restrict__ part) {
  __shared__ uint32_t key[kBlk];
  __shared__ int rid[kBlk + 1];     // run of each sorted position (-1 past the end)
  __shared__ int rstart[kBlk + 1];  // first sorted position of each run
  __shared__ int runid[kBlk];       // id of each run
  __shared__ int wtot[kBlkWaves];
  __shared__ double piece[kBlkWaves][64];  // a wave's unfinished last run
  const int t = threadIdx.x;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kBlk;
  const int nvalid = N - base < kBlk ? static_cast<int>(N - base) : kBlk;
  // Bitonic sort, thread t holding position t: at each step it keeps the
  // smaller or the larger of its key and its partner's (t ^ j), the smaller
  // when it is the lower of the two in an ascending stage.  Partners in the
  // same wave (j < 64) swap through cross-lane shuffles, the others through
  // LDS (two barriers per such step, 6 of the 45 steps).
  uint32_t kv = t < nvalid ? (static_cast<uint32_t>(clamp_tok(tok, base + t, vocab, err_flag)) << 9) |
                                 static_cast<uint32_t>(t)
                           : 0xFFFFFFFFu;
  for (int kk = 2; kk <= kBlk; kk <<= 1) {
    for (int j = kk >> 1; j > 0; j >>= 1) {
      uint32_t pv;
      if (j >= 64) {  // block-uniform branch
        key[t] = kv;
        __syncthreads();
        pv = key[t ^ j];
        __syncthreads();
      } else {
        pv = static_cast<uint32_t>(__shfl_xor(static_cast<int>(kv), j, 64));
      }
      const bool keep_min = ((t & j) == 0) == ((t & kk) == 0);
      kv = keep_min ? (kv < pv ? kv : pv) : (kv < pv ? pv : kv);
    }
  }
  key[t] = kv;
  __syncthreads();
  const uint32_t me = kv;
  const bool head = t < nvalid && (t == 0 || (key[t - 1] >> 9) != (me >> 9));
  int nrun = 0;
  const int before = block_excl_count(head, wtot, &nrun);
  rid[t] = t < nvalid ? (head ? before : before - 1) : -1;
  if (head) {
    rstart[before] = t;
    runid[before] = static_cast<int>(me >> 9);
    rid_out[base + before] = static_cast<int32_t>(me >> 9);
  }
  if (t == 0) {
    rid[kBlk] = -1;
    rstart[nrun] = nvalid;
  }
  __syncthreads();
  {  // the range index: fb[q] = the first run with an id of at least q kIdRange
     // (a binary search of the ascending run ids per q, the q spread over
     // the threads)
    int32_t *fb = first + static_cast<int64_t>(blockIdx.x) * (nq + 1);
    for (int64_t q = t; q <= nq; q += kBlk) {
      const int64_t target = q * kIdRange;
      int lo = 0, hi = nrun;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (runid[mid] < target)
          lo = mid + 1;
        else
          hi = mid;
      }
      fb[q] = lo;
    }
  }

  const int w = t >> 6, lane = t & 63;
  const int p0 = 64 * w;
  for (int j0 = 0; j0 < kp; j0 += 64) {  // the same trip count in every wave
    const int j = j0 + lane;
    const bool col = j < kp;
    const int jc = col ? j : kp - 1;
    // every load is issued (positions past the end read the last token's row)
    float v[64];
#pragma unroll
    for (int s2 = 0; s2 < 64; ++s2) {
      const int p = p0 + s2 < nvalid ? p0 + s2 : nvalid - 1;
      v[s2] = c32[(base + (key[p] & 511u)) * kp + jc];
    }
    // lane L describes position p0 + L: whether a run ends there (and its
    // run); the sequential sum below reads them as scalars
    const int pl = p0 + lane;
    const int rl = pl < nvalid ? rid[pl] : -1;
    const uint64_t ends = __ballot(pl < nvalid && rid[pl + 1] != rl);
    const uint64_t valid = __ballot(pl < nvalid);
    const int first_run = __shfl(rl, 0, 64);
    const bool first_open = nvalid > p0 && rstart[first_run > 0 ? first_run : 0] < p0;
    double acc = 0.0, tail = 0.0;
    int tail_run = -1;
    bool open = first_open;  // the current run began in an earlier wave
#pragma unroll
    for (int s2 = 0; s2 < 64; ++s2) {
      if ((valid >> s2) & 1) {
        acc += static_cast<double>(v[s2]);
        if ((ends >> s2) & 1) {  // the run ends here
          const int r = __builtin_amdgcn_readlane(rl, s2);
          if (!open) {
            if (col) part[((base + r) * kp) + j] = acc;
          } else {  // begun in an earlier wave: finished below
            tail = acc;
            tail_run = r;
          }
          acc = 0.0;
          open = false;
        } else if (s2 == 63) {  // continues into the next wave
          piece[w][lane] = acc;
        }
      }
    }
    __syncthreads();
    if (tail_run >= 0) {
      double tot = 0.0;
      for (int w2 = rstart[tail_run] >> 6; w2 < w; ++w2) tot += piece[w2][lane];
      tot += tail;
      if (col) part[((base + tail_run) * kp) + j] = tot;
    }
    __syncthreads();
  }
}

// One wave per id v: lane L takes block c0 + L (64 blocks per pass) and finds
// the block's run of id v by a binary search of the range index's runs
// (first[b][v / kIdRange] ..); the blocks that hold v are then visited in ascending order, 16 at a
// time (their loads issued together), lane j adding column j (64 columns per
// pass, KPC passes) in float64; gCS[v] += the total (ids that occur in no
// block are untouched).
template <int KPC>
__global__ __launch_bounds__(256) void id_merge_kernel(
    const int32_t *__restrict__ rid, const int32_t *__restrict__ first, int64_t nq, int64_t nblk,
    const double *__restrict__ part, int kp, int64_t k, int64_t vocab, float *__restrict__ gCS,
    int64_t ldgc) {
  const int lane = threadIdx.x & 63;
  const int64_t v = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (v >= vocab) return;
  const int64_t q = v / kIdRange;
  double acc[KPC];
#pragma unroll
  for (int c = 0; c < KPC; ++c) acc[c] = 0.0;
  bool any = false;
  for (int64_t c0 = 0; c0 < nblk; c0 += 64) {  // the same trip count in every lane
    const int64_t b = c0 + lane;
    int r = -1;
    if (b < nblk) {
      // the block's runs are in ascending id order: a binary search of the
      // range (a linear scan waits on one load per run, and the ranges of the
      // frequent ids hold tens of runs)
      const int32_t *fb = first + b * (nq + 1) + q;
      const int32_t *ids = rid + b * kBlk;
      int lo = fb[0], hi = fb[1];
      const int end = hi;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (ids[mid] < v)
          lo = mid + 1;
        else
          hi = mid;
      }
      if (lo < end && ids[lo] == v) r = lo;
    }
    uint64_t mask = __ballot(r >= 0);
    any = any || mask != 0;
    while (mask) {  // the blocks holding v, ascending, 16 at a time
      int64_t row[16];
      int cnt = 0;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        row[i] = 0;
        if (mask) {
          const int l = __builtin_ctzll(mask);
          mask &= mask - 1;
          row[i] = (c0 + l) * kBlk + __shfl(r, l, 64);
          ++cnt;
        }
      }
      double x[16][KPC];
#pragma unroll
      for (int i = 0; i < 16; ++i)
#pragma unroll
        for (int c = 0; c < KPC; ++c) {
          const int j = 64 * c + lane;
          x[i][c] = part[row[i] * kp + (j < kp ? j : kp - 1)];
        }
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (i < cnt)
#pragma unroll
          for (int c = 0; c < KPC; ++c) acc[c] += x[i][c];
    }
  }
  if (!any) return;
#pragma unroll
  for (int c = 0; c < KPC; ++c) {
    const int j = 64 * c + lane;
    if (j < k) gCS[v * ldgc + j] += static_cast<float>(acc[c]);
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
  double *part = reinterpret_cast<double *>(w + P.off_part);
  block_runs_kernel<<<dim3(static_cast<unsigned>(P.nblk)), kBlk, 0, s>>>(
      tok, N, vocab, err_flag, c32, static_cast<int>(P.kp), P.nq, I(P.off_rid), I(P.off_first),
      part);
  const dim3 mg(static_cast<unsigned>(ceil_div(vocab, 4)));
#define SN_MERGE(KPC)                                                                       \
  id_merge_kernel<KPC><<<mg, 256, 0, s>>>(I(P.off_rid), I(P.off_first), P.nq, P.nblk, part, \
                                          static_cast<int>(P.kp), L.k, vocab, gCS, ldgc)
  if (P.kp <= 64)
    SN_MERGE(1);
  else if (P.kp <= 128)
    SN_MERGE(2);
  else
    SN_MERGE(4);
#undef SN_MERGE
  return hipGetLastError();
}

}  // namespace sn
