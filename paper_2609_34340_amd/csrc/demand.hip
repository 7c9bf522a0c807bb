// vp_demand: routing -> per-expert counts -> demand rows (Sec. 3 model setup,
// one row copy per (token, expert) assignment), plus the stable (expert,
// token) order of one rank's assignments and its per-destination offsets
// (Sec. 5 buffer layout: the pack groups rows by destination).
//
// Kernels
//   hist_rows     one block per source rank; LDS-privatised histogram of its
//                 T*k expert ids, then the rank's demand row.
//   sort_count    one wavefront per chunk of the sorted rank's ids: per-chunk
//                 expert counts, written expert-major.
//   sort_scan     one block: exclusive scan of the expert-major counts, the
//                 destination offsets.
//   sort_scatter  one wavefront per chunk: stable within-chunk rank of every
//                 id from a wave-wide match mask built with one ballot per
//                 bit of the expert id, plus a prefix popcount.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace vp {
namespace {

constexpr int kChunk = 2048;          // ids per wavefront chunk of the counting sort
constexpr int kSortWaves = 4;         // wavefronts per block in sort_count / sort_scatter

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

// per-chunk expert counts, layout ccount[e * n_chunks + chunk]
__global__ void __launch_bounds__(64 * kSortWaves) sort_count(const int32_t* __restrict__ ids, int64_t Tk,
                                                              int32_t E, int32_t n_chunks,
                                                              int32_t* __restrict__ ccount) {
  extern __shared__ int32_t whist[];   // kSortWaves * E
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int chunk = blockIdx.x * kSortWaves + w;
  int32_t* h = whist + w * E;
  for (int e = lane; e < E; e += 64) h[e] = 0;
  wave_sync();
  if (chunk < n_chunks) {
    const int64_t b = (int64_t)chunk * kChunk, end = min(Tk, b + kChunk);
    for (int64_t x = b + lane; x < end; x += 64) {
      int e = ids[x];
      if ((unsigned)e < (unsigned)E) atomicAdd(&h[e], 1);
    }
    wave_sync();
    for (int e = lane; e < E; e += 64) ccount[(size_t)e * n_chunks + chunk] = h[e];
  }
}

// exclusive scan over E * n_chunks counts (expert-major) in one block
__global__ void __launch_bounds__(1024) sort_scan(int32_t* __restrict__ ccount, int64_t total, int32_t E,
                                                  int32_t N, int32_t n_chunks, int64_t* __restrict__ dest_off) {
  __shared__ int64_t wsum[16];
  __shared__ int64_t carry;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if (tid == 0) carry = 0;
  __syncthreads();
  const int eloc = E / N;
  for (int64_t b = 0; b < total; b += 1024) {
    const int64_t x = b + tid;
    int64_t v = x < total ? ccount[x] : 0;
    // inclusive wave scan
    int64_t s = v;
    for (int o = 1; o < 64; o <<= 1) {
      int64_t y = __shfl_up(s, o);
      if (lane >= o) s += y;
    }
    if (lane == 63) wsum[w] = s;
    __syncthreads();
    int64_t before = carry;
    for (int k = 0; k < w; ++k) before += wsum[k];
    const int64_t excl = before + s - v;
    if (x < total) {
      ccount[x] = (int32_t)excl;
      // the first chunk of expert j*eloc opens destination j
      if (x % n_chunks == 0) {
        const int64_t e = x / n_chunks;
        if (e % eloc == 0) dest_off[e / eloc] = excl;
      }
    }
    __syncthreads();
    if (tid == 1023) carry = excl + v;
    __syncthreads();
  }
  if (tid == 0) dest_off[N] = carry;
}

__global__ void __launch_bounds__(64 * kSortWaves) sort_scatter(const int32_t* __restrict__ ids, int64_t Tk,
                                                                int32_t k, int32_t E, int32_t n_chunks,
                                                                int32_t bits, const int32_t* __restrict__ coff,
                                                                int32_t* __restrict__ sorted_tok) {
  extern __shared__ int32_t run[];    // kSortWaves * E running positions
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int chunk = blockIdx.x * kSortWaves + w;
  if (chunk >= n_chunks) return;
  int32_t* pos = run + w * E;
  for (int e = lane; e < E; e += 64) pos[e] = coff[(size_t)e * n_chunks + chunk];
  wave_sync();
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int64_t b = (int64_t)chunk * kChunk, end = min(Tk, b + kChunk);
  for (int64_t x0 = b; x0 < end; x0 += 64) {
    const int64_t x = x0 + lane;
    const bool live = x < end;
    int e = live ? ids[x] : -1;
    const bool ok = live && (unsigned)e < (unsigned)E;
    // lanes holding the same expert id: AND of one ballot per id bit
    uint64_t same = __ballot(ok);
    for (int bt = 0; bt < bits; ++bt) {
      const uint64_t ones = __ballot(ok && ((e >> bt) & 1));
      same &= ((e >> bt) & 1) ? ones : ~ones;
    }
    int p = 0;
    if (ok) p = pos[e] + __popcll(same & lt);
    wave_sync();
    if (ok) {
      sorted_tok[p] = (int32_t)(x / k);
      if ((same & lt) == 0) pos[e] += __popcll(same);   // lowest lane of the group advances
    }
    wave_sync();
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
  const int blocks = (nch + kSortWaves - 1) / kSortWaves;
  const size_t lds = (size_t)kSortWaves * a.E * sizeof(int32_t);
  hipLaunchKernelGGL(sort_count, dim3(blocks), dim3(64 * kSortWaves), lds, s, ids, Tk, a.E, nch, ccount);
  hipLaunchKernelGGL(sort_scan, dim3(1), dim3(1024), 0, s, ccount, (int64_t)a.E * nch, a.E, a.N, nch,
                     a.dest_off);
  int bits = 0;
  while ((1 << bits) < a.E) ++bits;
  hipLaunchKernelGGL(sort_scatter, dim3(blocks), dim3(64 * kSortWaves), lds, s, ids, Tk, a.k, a.E, nch, bits,
                     ccount, a.sorted_tok);
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

}  // namespace vp
