// vp_demand: routing -> per-expert counts -> demand rows (Sec. 3 model setup,
// one row copy per (token, expert) assignment), plus the stable (expert,
// token) order of one rank's assignments and its per-destination offsets
// (Sec. 5 buffer layout: the pack groups rows by destination).
//
// Kernels
//   hist_rows     one block per source rank; LDS-privatised histogram of its
//                 T*k expert ids, then the rank's demand row.
//   sort_count    one block per 1024-id chunk of the sorted rank's ids:
//                 per-chunk expert counts, written expert-major.
//   sort_scan     one block: exclusive scan of the expert-major counts (one
//                 contiguous segment per thread), the destination offsets.
//   sort_scatter  one block per chunk: every id's stable rank inside its
//                 wave's 256 ids from a wave-wide match mask built with one
//                 ballot per bit of the expert id plus a prefix popcount,
//                 then the waves' counts scanned per expert.
//   control_words / receive_counts  the sparse expert-parallel control word
//                 of every (source, destination) pair from the counts, and
//                 its decode at the receiver.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace vp {
namespace {

constexpr int kSortThreads = 256;     // threads per block of the counting sort
constexpr int kPerThread = 4;         // ids per thread
constexpr int kChunk = kSortThreads * kPerThread;   // ids per block

__device__ inline void report(int32_t* status, int code) { atomicCAS(status, 0, code); }

__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__global__ void __launch_bounds__(1024) hist_rows(const int32_t* __restrict__ routing, int64_t Tk,
                                                  int32_t E, int32_t N, int32_t first_rank,
                                                  int64_t unit, int32_t* __restrict__ counts,
                                                  int64_t* __restrict__ demand, int32_t* status) {
  extern __shared__ int32_t hist[];
  const int r = blockIdx.x;
  for (int e = threadIdx.x; e < E; e += blockDim.x) hist[e] = 0;
  __syncthreads();
  const int32_t* row = routing + (size_t)r * Tk;
  bool bad = false;
  // 16-byte loads of four ids where the row is 16-byte aligned
  const int64_t nv = ((((uintptr_t)row) & 15) == 0) ? Tk / 4 : 0;
  const int4* row4 = (const int4*)row;
  for (int64_t v = threadIdx.x; v < nv; v += blockDim.x) {
    int4 q = row4[v];
    int ids[4] = {q.x, q.y, q.z, q.w};
    for (int m = 0; m < 4; ++m) {
      if ((unsigned)ids[m] < (unsigned)E) atomicAdd(&hist[ids[m]], 1);
      else bad = true;
    }
  }
  for (int64_t x = nv * 4 + threadIdx.x; x < Tk; x += blockDim.x) {
    int e = row[x];
    if ((unsigned)e < (unsigned)E) atomicAdd(&hist[e], 1);
    else bad = true;
  }
  if (bad) report(status, VP_ERR_INVALID_ARGUMENT);
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) counts[(size_t)r * E + e] = hist[e];
  const int eloc = E / N, self = first_rank + r;
  for (int j = threadIdx.x; j < N; j += blockDim.x) {
    int64_t c = 0;
    for (int e = j * eloc; e < (j + 1) * eloc; ++e) c += hist[e];
    demand[(size_t)r * N + j] = j == self ? 0 : c * unit;
  }
}

// Counting sort of one rank's ids, chunks of kChunk ids, one block per
// chunk.  Counts are laid out ccount[e * n_chunks + chunk].
__global__ void __launch_bounds__(kSortThreads) sort_count(const int32_t* __restrict__ ids, int64_t Tk,
                                                          int32_t E, int32_t n_chunks,
                                                          int32_t* __restrict__ ccount) {
  extern __shared__ int32_t h[];   // E
  const int tid = threadIdx.x, chunk = blockIdx.x;
  for (int e = tid; e < E; e += kSortThreads) h[e] = 0;
  __syncthreads();
  const int64_t b = (int64_t)chunk * kChunk;
  int ev[kPerThread];
#pragma unroll
  for (int m = 0; m < kPerThread; ++m) {
    const int64_t x = b + tid + m * kSortThreads;
    ev[m] = x < Tk ? ids[x] : -1;
  }
#pragma unroll
  for (int m = 0; m < kPerThread; ++m)
    if ((unsigned)ev[m] < (unsigned)E) atomicAdd(&h[ev[m]], 1);
  __syncthreads();
  for (int e = tid; e < E; e += kSortThreads) ccount[(size_t)e * n_chunks + chunk] = h[e];
}

// Exclusive scan of the E * n_chunks counts (expert-major) in one block:
// tiles of 4096 counts, each thread a coalesced run of four, up to eight
// tiles loaded ahead.  Counts and offsets fit 32 bits (at most T*k).
__global__ void __launch_bounds__(1024) sort_scan(int32_t* __restrict__ ccount, int64_t total, int32_t E,
                                                  int32_t N, int32_t n_chunks, int64_t* __restrict__ dest_off) {
  constexpr int V = 4, TB = 8;
  __shared__ int32_t wsum[16];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int32_t carry = 0;
  const bool vec = (((uintptr_t)ccount) & 15) == 0;
  for (int64_t b0 = 0; b0 < total; b0 += (int64_t)1024 * V * TB) {
    int32_t v[TB][V];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      const int64_t x = b0 + ((int64_t)tb * 1024 + tid) * V;
      if (vec && x + V <= total) {
        const int4 q = *(const int4*)(ccount + x);
        v[tb][0] = q.x; v[tb][1] = q.y; v[tb][2] = q.z; v[tb][3] = q.w;
      } else {
#pragma unroll
        for (int m = 0; m < V; ++m) v[tb][m] = x + m < total ? ccount[x + m] : 0;
      }
    }
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      const int64_t x = b0 + ((int64_t)tb * 1024 + tid) * V;
      if (b0 + (int64_t)tb * 1024 * V >= total) break;   // uniform
      const int32_t mine = v[tb][0] + v[tb][1] + v[tb][2] + v[tb][3];
      int32_t s = mine;
      for (int o = 1; o < 64; o <<= 1) {
        const int32_t y = __shfl_up(s, o);
        if (lane >= o) s += y;
      }
      if (lane == 63) wsum[w] = s;
      __syncthreads();
      int32_t run = carry + s - mine, all = 0;
      for (int u = 0; u < 16; ++u) {
        if (u < w) run += wsum[u];
        all += wsum[u];
      }
#pragma unroll
      for (int m = 0; m < V; ++m) {
        if (x + m < total) ccount[x + m] = run;
        run += v[tb][m];
      }
      carry += all;
      __syncthreads();
    }
  }
  __syncthreads();
  // destination j opens at the first chunk of expert j*eloc
  const int eloc = E / N;
  for (int j = tid; j < N; j += 1024) dest_off[j] = ccount[(size_t)j * eloc * n_chunks];
  if (tid == 0) dest_off[N] = carry;
}

// Stable scatter of one chunk: wave v ranks the ids [v*64*kPerThread, ...)
// of the chunk with one ballot per id bit (a match mask) and a prefix
// popcount; the waves' counts are then scanned per expert.
__global__ void __launch_bounds__(kSortThreads) sort_scatter(const int32_t* __restrict__ ids, int64_t Tk,
                                                            int32_t k, int32_t E, int32_t n_chunks,
                                                            int32_t bits, const int32_t* __restrict__ coff,
                                                            int32_t* __restrict__ sorted_tok,
                                                            uint8_t* __restrict__ sorted_slot) {
  extern __shared__ int32_t wc[];    // [kSortThreads / 64][E]
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, chunk = blockIdx.x;
  constexpr int kW = kSortThreads / 64;
  const int64_t base = (int64_t)chunk * kChunk + (int64_t)w * 64 * kPerThread;
  int ev[kPerThread];
#pragma unroll
  for (int m = 0; m < kPerThread; ++m) {
    const int64_t x = base + m * 64 + lane;
    ev[m] = x < Tk ? ids[x] : -1;
  }
  int32_t* mine = wc + w * E;
  for (int e = lane; e < E; e += 64) mine[e] = 0;
  wave_sync();
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int rk[kPerThread];
#pragma unroll
  for (int m = 0; m < kPerThread; ++m) {
    const int e = ev[m];
    const bool ok = (unsigned)e < (unsigned)E;
    uint64_t same = __ballot(ok);
    for (int bt = 0; bt < bits; ++bt) {
      const uint64_t ones = __ballot(ok && ((e >> bt) & 1));
      same &= ((e >> bt) & 1) ? ones : ~ones;
    }
    rk[m] = ok ? mine[e] + __popcll(same & lt) : 0;
    wave_sync();
    if (ok && (same & lt) == 0) mine[e] += __popcll(same);   // lowest lane of the group advances
    wave_sync();
  }
  __syncthreads();
  for (int e = tid; e < E; e += kSortThreads) {
    int32_t acc = coff[(size_t)e * n_chunks + chunk];
    for (int v = 0; v < kW; ++v) {
      const int32_t c = wc[v * E + e];
      wc[v * E + e] = acc;
      acc += c;
    }
  }
  __syncthreads();
#pragma unroll
  for (int m = 0; m < kPerThread; ++m) {
    const int e = ev[m];
    if ((unsigned)e < (unsigned)E) {
      const int64_t x = base + m * 64 + lane, t = x / k;
      sorted_tok[mine[e] + rk[m]] = (int32_t)t;
      if (sorted_slot) sorted_slot[mine[e] + rk[m]] = (uint8_t)(x - t * k);
    }
  }
}

__global__ void demand_heads_kernel(int64_t T, const int64_t* __restrict__ head_lo, int64_t head_bytes,
                                    int32_t N, int32_t first_rank, int64_t* __restrict__ demand,
                                    int32_t* status) {
  const int r = blockIdx.x;
  for (int j = threadIdx.x; j < N; j += blockDim.x) {
    const int64_t h = head_lo[j + 1] - head_lo[j];
    if (h < 0) report(status, VP_ERR_INVALID_ARGUMENT);
    demand[(size_t)r * N + j] = (j == first_rank + r || h < 0) ? 0 : T * h * head_bytes;
  }
}

// Sparse expert-parallel control words (Sec. 5): one thread per (source row,
// destination) pair.  The destination's L local experts are L consecutive
// counts of the row: bit l marks an expert with rows, the bits above L carry
// the count of the highest such expert (the last payload of the pair's
// expert-ascending stream).  The self pair and pairs without rows get 0.
__global__ void __launch_bounds__(256) control_words_kernel(const int32_t* __restrict__ counts, int32_t R,
                                                            int32_t E, int32_t N, int32_t L, int32_t first_rank,
                                                            uint32_t* __restrict__ words, int32_t* status) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= (int64_t)R * N) return;
  const int r = (int)(p / N), j = (int)(p - (int64_t)r * N);
  const int32_t* c = counts + (size_t)r * E + (size_t)j * L;
  uint32_t bitmap = 0;
  int32_t last = 0;
  bool bad = false;
  for (int l = 0; l < L; ++l) {
    const int32_t v = c[l];
    bad |= v < 0;
    if (v > 0) {
      bitmap |= 1u << l;
      last = v;
    }
  }
  uint32_t w = 0;
  if (bad) {
    report(status, VP_ERR_INVALID_ARGUMENT);
  } else if (j != first_rank + r && bitmap != 0) {
    if (((uint64_t)last >> (32 - L)) != 0) report(status, VP_ERR_CAPACITY);   // 32 - L count bits
    else w = bitmap | ((uint32_t)last << L);
  }
  words[p] = w;
}

// The receiver's side: one thread per (source, local expert).  A clear bitmap
// bit means no rows; the designated (highest active) expert's count is in the
// word; the other active experts' counts come from their signals.
__global__ void __launch_bounds__(256) receive_counts_kernel(const uint32_t* __restrict__ words,
                                                             int64_t word_stride,
                                                             const int32_t* __restrict__ signal, int32_t N,
                                                             int32_t L, int32_t* __restrict__ counts) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= (int64_t)N * L) return;
  const int i = (int)(p / L), l = (int)(p - (int64_t)i * L);
  const uint32_t w = words[(size_t)i * word_stride];
  const uint32_t bitmap = w & ((1u << L) - 1);
  int32_t c = 0;
  if (bitmap >> l & 1) c = (31 - __builtin_clz(bitmap)) == l ? (int32_t)(w >> L) : signal[p];
  counts[p] = c;
}

int n_chunks_of(int64_t Tk) { return (int)((Tk + kChunk - 1) / kChunk); }

}  // namespace

size_t demand_workspace(int64_t T, int32_t k, int32_t E) {
  const int64_t Tk = T * k;
  return (size_t)E * (size_t)std::max(1, n_chunks_of(Tk)) * sizeof(int32_t);
}

vp_status launch_demand(const DemandLaunch& a, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const int64_t Tk = a.T * a.k;
  hipLaunchKernelGGL(hist_rows, dim3(a.R), dim3(1024), (size_t)a.E * sizeof(int32_t), s, a.routing, Tk, a.E,
                     a.N, a.first_rank, a.unit, a.counts, a.demand, a.status);
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "hist_rows launch failed");
  if (a.sort_row < 0) return VP_OK;
  const int32_t* ids = a.routing + (size_t)a.sort_row * Tk;
  const int nch = std::max(1, n_chunks_of(Tk));
  int32_t* ccount = (int32_t*)a.ws;
  hipLaunchKernelGGL(sort_count, dim3(nch), dim3(kSortThreads), (size_t)a.E * sizeof(int32_t), s, ids, Tk, a.E,
                     nch, ccount);
  hipLaunchKernelGGL(sort_scan, dim3(1), dim3(1024), 0, s, ccount, (int64_t)a.E * nch, a.E, a.N, nch,
                     a.dest_off);
  int bits = 0;
  while ((1 << bits) < a.E) ++bits;
  hipLaunchKernelGGL(sort_scatter, dim3(nch), dim3(kSortThreads), (size_t)(kSortThreads / 64) * a.E * sizeof(int32_t),
                     s, ids, Tk, a.k, a.E, nch, bits, ccount, a.sorted_tok, a.sorted_slot);
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "sort launch failed");
  return VP_OK;
}

vp_status launch_demand_heads(int64_t T, const int64_t* head_lo, int64_t head_bytes, int32_t N,
                              int32_t first_rank, int32_t R, int64_t* demand, int32_t* status,
                              void* stream) {
  hipStream_t s = (hipStream_t)stream;
  hipLaunchKernelGGL(demand_heads_kernel, dim3(R), dim3(256), 0, s, T, head_lo, head_bytes, N, first_rank,
                     demand, status);
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "demand_heads launch failed");
  return VP_OK;
}

vp_status launch_control_words(const int32_t* counts, int32_t R, int32_t E, int32_t N, int32_t first_rank,
                               uint32_t* words, int32_t* status, void* stream) {
  const int64_t n = (int64_t)R * N;
  if (n == 0) return VP_OK;
  hipLaunchKernelGGL(control_words_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, (hipStream_t)stream,
                     counts, R, E, N, E / N, first_rank, words, status);
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "control_words launch failed");
  return VP_OK;
}

vp_status launch_receive_counts(const uint32_t* words, int64_t word_stride, const int32_t* signal, int32_t N,
                                int32_t L, int32_t* counts, void* stream) {
  const int64_t n = (int64_t)N * L;
  hipLaunchKernelGGL(receive_counts_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                     (hipStream_t)stream, words, word_stride, signal, N, L, counts);
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "receive_counts launch failed");
  return VP_OK;
}

}  // namespace vp
