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
//           epilogue), then a deterministic segmented sum by token id:
//           a one-workgroup stable counting sort of the token indices
//           (segments of equal ids, indices ascending), per-chunk sums of at
//           most 64 rows of a segment, and per-segment sums of its chunks,
//           every sum in a fixed order in float64.
#include "sn_device.h"
#include "sn_internal.h"

namespace sn {

namespace {

constexpr int kSortThreads = 1024;

__device__ __forceinline__ int64_t ceil_div_dev(int64_t a, int64_t b) { return (a + b - 1) / b; }
constexpr int kChunk = 64;  // rows per chunk of a segment

struct EmbedPlan {
  int64_t kp = 0, maxseg = 0, maxchunk = 0;
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
  auto ints = [&](size_t &o, int64_t n) {
    o = off;
    off = align256(off + static_cast<size_t>(n) * 4);
  };
  ints(P.off_cnt, vocab);
  ints(P.off_cur, vocab);
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

// One workgroup: counting sort of the token indices by (clamped) id, stable,
// and the segment and chunk tables.  meta[0] = segments, meta[1] = chunks.
__global__ __launch_bounds__(kSortThreads) void sort_kernel(
    const int32_t *__restrict__ tok, int64_t N, int64_t vocab, int32_t *err_flag,
    int32_t *__restrict__ cnt, int32_t *__restrict__ cur, int32_t *__restrict__ order,
    int32_t *__restrict__ seg_id, int32_t *__restrict__ seg_off, int32_t *__restrict__ seg_ch,
    int32_t *__restrict__ cbeg, int32_t *__restrict__ cend, int32_t *__restrict__ meta) {
  __shared__ int buf[kSortThreads];
  __shared__ int sid[kSortThreads];
  const int t = threadIdx.x;
  const int nt = kSortThreads;
  auto id_of = [&](int64_t i) {
    int64_t v = tok[i];
    if (v < 0 || v >= vocab) {
      if (err_flag) atomicOr(err_flag, 1);
      v = v < 0 ? 0 : vocab - 1;
    }
    return static_cast<int>(v);
  };
  // 1. histogram of the ids
  for (int64_t v = t; v < vocab; v += nt) cnt[v] = 0;
  __threadfence();
  __syncthreads();
  for (int64_t i = t; i < N; i += nt) atomicAdd(&cnt[id_of(i)], 1);
  __threadfence();
  __syncthreads();
  // 2. offsets of the ids (thread t: ids [v0, v1)) and the segments (ids that occur)
  const int64_t per = ceil_div_dev(vocab, nt);
  const int64_t v0 = t * per < vocab ? t * per : vocab;
  const int64_t v1 = v0 + per < vocab ? v0 + per : vocab;
  int sum = 0, nz = 0;
  for (int64_t v = v0; v < v1; ++v) {
    sum += cnt[v];
    nz += cnt[v] > 0;
  }
  int total, nseg;
  int run = block_excl_scan(sum, buf, &total);
  int seg = block_excl_scan(nz, buf, &nseg);
  for (int64_t v = v0; v < v1; ++v) {
    const int c = cnt[v];
    cur[v] = run;
    if (c > 0) {
      seg_id[seg] = static_cast<int>(v);
      seg_off[seg] = run;
      ++seg;
    }
    run += c;
  }
  if (t == 0) {
    seg_off[nseg] = static_cast<int>(N);
    meta[0] = nseg;
  }
  __threadfence();
  __syncthreads();
  // 3. stable placement, 1024 tokens at a time: a token's slot is its id's
  // cursor plus the number of earlier tokens of the chunk with the same id;
  // the id's last token of the chunk advances the cursor
  for (int64_t c0 = 0; c0 < N; c0 += nt) {
    const int64_t i = c0 + t;
    const int v = i < N ? id_of(i) : -1;
    sid[t] = v;
    __syncthreads();
    int rank = 0;
    bool last = true;
    if (v >= 0) {
      for (int j = 0; j < t; ++j) rank += sid[j] == v;
      for (int j = t + 1; j < nt; ++j) last = last && sid[j] != v;
      order[cur[v] + rank] = static_cast<int>(i);
    }
    __syncthreads();
    if (v >= 0 && last) cur[v] += rank + 1;
    __threadfence();
    __syncthreads();
  }
  // 4. chunks of at most kChunk rows per segment (thread t: segments [s0, s1))
  const int64_t sper = ceil_div_dev(nseg, nt);
  const int64_t s0 = t * sper < nseg ? t * sper : nseg;
  const int64_t s1 = s0 + sper < nseg ? s0 + sper : nseg;
  int nch = 0;
  for (int64_t s = s0; s < s1; ++s) nch += (seg_off[s + 1] - seg_off[s] + kChunk - 1) / kChunk;
  int nchunk;
  int q = block_excl_scan(nch, buf, &nchunk);
  for (int64_t s = s0; s < s1; ++s) {
    seg_ch[s] = q;
    for (int b = seg_off[s]; b < seg_off[s + 1]; b += kChunk) {
      cbeg[q] = b;
      cend[q] = b + kChunk < seg_off[s + 1] ? b + kChunk : seg_off[s + 1];
      ++q;
    }
  }
  if (t == 0) {
    seg_ch[nseg] = nchunk;
    meta[1] = nchunk;
  }
}

// One wave per chunk: part[q][j] = sum over the chunk's rows (ascending
// token index) of c32[row][j], float64.
__global__ __launch_bounds__(256) void chunk_sum_kernel(const float *__restrict__ c32, int64_t kp,
                                                        const int32_t *__restrict__ order,
                                                        const int32_t *__restrict__ cbeg,
                                                        const int32_t *__restrict__ cend,
                                                        const int32_t *__restrict__ meta,
                                                        double *__restrict__ part) {
  const int lane = threadIdx.x & 63;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (q >= meta[1]) return;
  const int b = cbeg[q], e = cend[q];
  for (int64_t j = lane; j < kp; j += 64) {
    double acc = 0.0;
    for (int p = b; p < e; ++p) acc += static_cast<double>(c32[static_cast<int64_t>(order[p]) * kp + j]);
    part[q * kp + j] = acc;
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
  sort_kernel<<<dim3(1), kSortThreads, 0, s>>>(tok, N, vocab, err_flag, I(P.off_cnt), I(P.off_cur),
                                                I(P.off_order), I(P.off_segid), I(P.off_segoff),
                                                I(P.off_segch), I(P.off_cbeg), I(P.off_cend),
                                                I(P.off_meta));
  double *part = reinterpret_cast<double *>(w + P.off_part);
  chunk_sum_kernel<<<dim3(static_cast<unsigned>(ceil_div(P.maxchunk, 4))), 256, 0, s>>>(
      c32, P.kp, I(P.off_order), I(P.off_cbeg), I(P.off_cend), I(P.off_meta), part);
  seg_sum_kernel<<<dim3(static_cast<unsigned>(ceil_div(P.maxseg, 4))), 256, 0, s>>>(
      part, P.kp, L.k, I(P.off_segid), I(P.off_segch), I(P.off_meta), gCS, ldgc);
  return hipGetLastError();
}

}  // namespace sn
