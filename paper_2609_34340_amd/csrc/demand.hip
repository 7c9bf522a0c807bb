// vp_demand: routing -> per-expert counts -> demand rows (Sec. 3 model setup,
// one row copy per (token, expert) assignment), plus the stable (expert,
// token) order of one rank's assignments and its per-destination offsets
// (Sec. 5 buffer layout: the pack groups rows by destination).
//
// Kernels
//   demand_count   pass 1: every row's ids split over many workgroups, each
//                  counting its part in per-wavefront LDS histograms and
//                  writing the part's expert counts; the same launch counts
//                  the sorted row per 2048-id chunk (expert-major).
//   sort_scan      only for sorted rows of more than 64 chunks: one
//                  workgroup turns the chunk counts into offsets.
//   demand_finish  pass 2: one workgroup per row sums its parts (at most
//                  16 per row for rows up to 131,072 ids: one round of
//                  loads) into the row's counts and demand row; one
//                  workgroup per sort chunk (512 threads, four ids each,
//                  for up to 256 experts) places its ids: a stable rank
//                  inside each wave's ids from a match mask built with one
//                  ballot per bit of the expert id plus a prefix popcount,
//                  while the chunk counts it needs are in flight; then the
//                  chunk's offsets from all chunk counts (expert totals, a
//                  block scan, the earlier chunks' counts) and the waves'
//                  counts scanned per expert.  Loads are unconditional
//                  (clamped indexes, masked results) so that each wait
//                  covers only the load it needs.
//   No workgroup waits for another: the kernel boundary publishes pass 1.
//   control_words / receive_counts  the sparse expert-parallel control word
//                 of every (source, destination) pair from the counts, and
//                 its decode at the receiver.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace vp {
namespace {

constexpr int kThreads = 256;                    // threads of every demand workgroup
constexpr int kWaves = kThreads / 64;
constexpr int kChunk = 2048;                     // ids per sort chunk
constexpr int kInBlockScan = 64;                 // sort chunks up to which each scatter
                                                 // workgroup derives its own offsets

__device__ inline void report(int32_t* status, int code) { atomicCAS(status, 0, code); }

__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

struct DemandArgs {
  const int32_t* routing;
  int64_t Tk, part, unit;
  int32_t E, N, first_rank, R, P, sort_row, nch, nch4, k, bits;
  uint64_t k_magic;     // ceil(2^40 / k): token of assignment x = mulhi(x << 24, k_magic)
  bool scanned;         // a scan kernel has turned the chunk counts into offsets
  int32_t* counts;
  int64_t* demand;
  int32_t* sorted_tok;
  uint8_t* sorted_slot;
  int64_t* dest_off;
  int32_t* partials;    // [R][P][E] expert counts of each part of each row
  int32_t* ccount;      // [E][nch4] counts of the sorted row's chunks (zero past nch)
  int32_t* status;
};

// Counts the ids [lo, hi) into an LDS histogram (16-byte loads of four ids
// where the range is aligned, four loads in flight per thread).
__device__ inline void count_ids(const int32_t* __restrict__ ids, int64_t lo, int64_t hi, int32_t E,
                                 int32_t* hist, bool& bad) {
  int64_t v1 = lo;
  if ((((uintptr_t)(ids + lo)) & 15) == 0) v1 = lo + (hi - lo) / 4 * 4;
  const int4* q4 = (const int4*)(ids + lo);
  const int64_t nv = (v1 - lo) / 4;
  for (int64_t v = threadIdx.x; v < nv; v += 4 * kThreads) {
    int4 q[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (v + u * kThreads < nv) q[u] = q4[v + u * kThreads];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (v + u * kThreads >= nv) break;
      const int e4[4] = {q[u].x, q[u].y, q[u].z, q[u].w};
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        if ((unsigned)e4[m] < (unsigned)E) atomicAdd(&hist[e4[m]], 1);
        else bad = true;
      }
    }
  }
  for (int64_t x = v1 + threadIdx.x; x < hi; x += kThreads) {
    const int e = ids[x];
    if ((unsigned)e < (unsigned)E) atomicAdd(&hist[e], 1);
    else bad = true;
  }
}

// Pass 1.  Workgroups [0, nsort) count the sorted row's 2048-id chunks
// (expert-major, the last one also zeroes the padding up to nch4);
// workgroups after them count one part of one row each.  Every workgroup
// keeps one LDS histogram per wavefront.
__global__ void __launch_bounds__(kThreads) demand_count(DemandArgs a) {
  extern __shared__ int32_t sh[];   // kWaves * E
  const int tid = threadIdx.x, w = tid >> 6, E = a.E;
  const int nsort = a.sort_row >= 0 ? a.nch : 0;
  const int b = blockIdx.x;
  const bool sort_blk = b < nsort;
  int r, p;
  int64_t lo;
  if (sort_blk) {
    r = a.sort_row;
    p = b;
    lo = (int64_t)p * kChunk;
  } else {
    r = (b - nsort) / a.P;
    p = (b - nsort) - r * a.P;
    lo = (int64_t)p * a.part;
  }
  const int64_t hi = min(a.Tk, lo + (sort_blk ? (int64_t)kChunk : a.part));
  lo = min(lo, hi);
  for (int e = tid; e < kWaves * E; e += kThreads) sh[e] = 0;
  __syncthreads();
  bool bad = false;
  count_ids(a.routing + (size_t)r * a.Tk, lo, hi, E, sh + w * E, bad);
  if (bad && !sort_blk) report(a.status, VP_ERR_INVALID_ARGUMENT);
  __syncthreads();
  for (int e = tid; e < E; e += kThreads) {
    int32_t c = 0;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) c += sh[v * E + e];
    if (sort_blk) {
      int32_t* q = a.ccount + (size_t)e * a.nch4;
      q[p] = c;
      if (p == a.nch - 1)
        for (int x = a.nch; x < a.nch4; ++x) q[x] = 0;
    } else {
      a.partials[((size_t)r * a.P + p) * E + e] = c;
    }
  }
}

// One workgroup scans all chunk counts (expert-major) into offsets, for
// sorted rows of more than kInBlockScan chunks: tiles of 4096 counts, each
// thread a coalesced run of four, eight tiles loaded ahead.
__global__ void __launch_bounds__(1024) sort_scan(int32_t* __restrict__ ccount, int64_t total, int32_t E,
                                                  int32_t N, int32_t nch4, int64_t* __restrict__ dest_off) {
  constexpr int V = 4, TB = 8;
  __shared__ int32_t wsum[16];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int32_t carry = 0;
  for (int64_t b0 = 0; b0 < total; b0 += (int64_t)1024 * V * TB) {
    int32_t v[TB][V];
#pragma unroll
    for (int tb = 0; tb < TB; ++tb) {
      const int64_t x = b0 + ((int64_t)tb * 1024 + tid) * V;
      if (x + V <= total) {
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
  for (int j = tid; j < N; j += 1024) dest_off[j] = ccount[(size_t)j * eloc * nch4];
  if (tid == 0) dest_off[N] = carry;
}

// Exclusive scan over the block of n values in LDS (n <= 16 * TH): each
// thread a contiguous run; returns the total.
template <int TH>
__device__ inline int32_t block_excl_scan(int32_t* v, int n, int32_t* wtot) {
  constexpr int W = TH / 64;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int per = (n + TH - 1) / TH;
  const int e0 = min(n, tid * per), e1 = min(n, e0 + per);
  int32_t own = 0;
  for (int e = e0; e < e1; ++e) own += v[e];
  int32_t incl = own;
  for (int o = 1; o < 64; o <<= 1) {
    const int32_t y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == 63) wtot[w] = incl;
  __syncthreads();
  int32_t run = incl - own, all = 0;
  for (int u = 0; u < W; ++u) {
    if (u < w) run += wtot[u];
    all += wtot[u];
  }
  for (int e = e0; e < e1; ++e) {
    const int32_t x = v[e];
    v[e] = run;
    run += x;
  }
  __syncthreads();
  return all;
}

// Pass 2.  Workgroup c < nch places the ids of sort chunk c; the R
// workgroups after them merge their row's parts into its counts and demand
// row.  A chunk's offsets: expert e starts at the total of the experts below
// e plus the counts of e in the chunks before c (each workgroup reads every
// chunk count, or the scan kernel's offsets for long rows).  Inside the
// chunk, wave v ranks its ids with one ballot per id bit (a match mask) and
// a prefix popcount; the waves' counts are then scanned per expert.
// Offsets of a sort chunk: from the scan kernel, or from every chunk's
// counts (at most kInBlockScan chunks) held in registers (up to 256
// experts, TH / 256 threads per expert) or reloaded.  TH threads per
// workgroup, kChunk / TH ids per thread.
enum { kOffScanned = 0, kOffHeld = 1, kOffReload = 2 };

template <int OFF, int TH>
__global__ void __launch_bounds__(TH) demand_finish(DemandArgs a) {
  constexpr int kW = TH / 64;                       // waves
  constexpr int kPT = kChunk / TH;                  // ids per thread of a sort chunk
  constexpr int kSplit = TH / 256;                  // threads per expert holding its chunk counts
  constexpr int kC4 = kInBlockScan / 4 / kSplit;    // chunk counts per thread, in fours
  static_assert(kPT * TH == kChunk && kSplit >= 1 && kC4 * 4 * kSplit == kInBlockScan, "block shape");
  extern __shared__ int32_t sh[];   // rows: E; chunks: off [E], tot [E], wc [kW][E]
  __shared__ int32_t wtot[kW];
  const int tid = threadIdx.x, E = a.E;
  // the sort chunks, whose ranking is the longest work, come first
  const int nsort = a.sort_row >= 0 ? a.nch : 0;
  const int b = blockIdx.x;
  if (b >= nsort) {
    const int r = b - nsort;
    const int32_t* q = a.partials + (size_t)r * a.P * E;
    for (int e = tid; e < E; e += TH) {
      // loads of 16 parts issued together, then summed
      int32_t c = 0;
      for (int pp = 0; pp < a.P; pp += 16) {
        int32_t v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) v[u] = pp + u < a.P ? q[(size_t)(pp + u) * E + e] : 0;
#pragma unroll
        for (int u = 0; u < 16; ++u) c += v[u];
      }
      a.counts[(size_t)r * E + e] = c;
      sh[e] = c;
    }
    __syncthreads();
    const int eloc = E / a.N, self = a.first_rank + r;
    for (int j = tid; j < a.N; j += TH) {
      int64_t c = 0;
      for (int e = j * eloc; e < (j + 1) * eloc; ++e) c += sh[e];
      a.demand[(size_t)r * a.N + j] = j == self ? 0 : c * a.unit;
    }
    return;
  }
  const int chunk = b;
  const int lane = tid & 63, w = tid >> 6;
  int32_t* off = sh;
  int32_t* tot = sh + E;
  int32_t* wc = sh + 2 * E;
  const int32_t* ids = a.routing + (size_t)a.sort_row * a.Tk;
  if (a.Tk <= 0) {   // an empty row: every destination's range is empty
    if (chunk == 0)
      for (int j = tid; j <= a.N; j += TH) a.dest_off[j] = 0;
    return;
  }
  // the chunk's ids first, then its chunk counts, all loads unconditional
  // (indexes clamped into range, results masked after) so that the ranking
  // below waits for the ids only and the counts' latency hides behind it
  const int64_t base = (int64_t)chunk * kChunk + (int64_t)w * 64 * kPT;
  int ev[kPT];
#pragma unroll
  for (int m = 0; m < kPT; ++m) {
    const int64_t x = base + m * 64 + lane;
    ev[m] = ids[x < a.Tk ? x : a.Tk - 1];
  }
  // The chunk counts: the scan kernel's offsets, or the counts of the
  // thread's share of every chunk of its expert (at most kInBlockScan
  // chunks) held in registers through the ranking, which does not depend on
  // them.
  const int he = tid / kSplit, c4lo = (tid % kSplit) * kC4;   // held: expert, first four of the share
  int4 cv[kC4];
  if (OFF == kOffScanned) {
    for (int e = tid; e < E; e += TH) off[e] = a.ccount[(size_t)e * a.nch4 + chunk];
  } else if (OFF == kOffHeld) {
    const int n4 = a.nch4 / 4;
    const int4* q = (const int4*)(a.ccount + (size_t)(he < E ? he : 0) * a.nch4);
#pragma unroll
    for (int c = 0; c < kC4; ++c) cv[c] = q[c4lo + c < n4 ? c4lo + c : n4 - 1];
  }
  int32_t* mine = wc + w * E;
  for (int e = lane; e < E; e += 64) mine[e] = 0;
  wave_sync();
  // Match masks of all kPT ids at once, bit by bit of the expert id: the kPT
  // ballots of one bit are independent, so their latencies overlap.  Ids
  // past the row (and bad ids) are no ids.
  uint64_t same[kPT];
#pragma unroll
  for (int m = 0; m < kPT; ++m) {
    if (base + m * 64 + lane >= a.Tk) ev[m] = -1;
    same[m] = __ballot((unsigned)ev[m] < (unsigned)E);
  }
  for (int bt = 0; bt < a.bits; ++bt) {
#pragma unroll
    for (int m = 0; m < kPT; ++m) {
      const bool one = ((uint32_t)ev[m] >> bt) & 1u;
      const uint64_t ones = __ballot(one);
      same[m] &= one ? ones : ~ones;
    }
  }
  // The wave's running count of each expert: id m's rank is the count before
  // it plus its lower lanes with the same expert; the lowest lane of each
  // group then adds the group's size.  The adds return nothing and the
  // wave's LDS operations complete in order, so no id waits for the one
  // before it; the counts read are summed after the last add.
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int rk[kPT], cnt_before[kPT];
#pragma unroll
  for (int m = 0; m < kPT; ++m) {
    const int e = ev[m];
    const bool ok = (unsigned)e < (unsigned)E;
    const uint64_t below = same[m] & lt;
    rk[m] = __popcll(below);
    cnt_before[m] = mine[ok ? e : 0];
    wave_sync();
    if (ok && below == 0)
      __hip_atomic_fetch_add(&mine[e], (int32_t)__popcll(same[m]), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
    wave_sync();
  }
#pragma unroll
  for (int m = 0; m < kPT; ++m) rk[m] += cnt_before[m];
  if (OFF != kOffScanned) {
    if (OFF == kOffHeld) {
      const int n4 = a.nch4 / 4;
      int32_t all = 0, before = 0;
#pragma unroll
      for (int c = 0; c < kC4; ++c) {
        // the clamped loads past the last chunk count nothing
        const int c4 = c4lo + c;
        const bool in = c4 < n4;
        const int32_t x4[4] = {in ? cv[c].x : 0, in ? cv[c].y : 0, in ? cv[c].z : 0, in ? cv[c].w : 0};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          all += x4[q];
          before += 4 * c4 + q < chunk ? x4[q] : 0;
        }
      }
#pragma unroll
      for (int o = 1; o < kSplit; o <<= 1) {   // the expert's threads are neighbouring lanes
        all += __shfl_xor(all, o);
        before += __shfl_xor(before, o);
      }
      if (he < E && tid % kSplit == 0) {
        tot[he] = all;
        off[he] = before;
      }
    } else {
      for (int e = tid; e < E; e += TH) {
        const int4* q = (const int4*)(a.ccount + (size_t)e * a.nch4);
        const int n4 = a.nch4 / 4;
        int4 v[kInBlockScan / 4];
#pragma unroll
        for (int c4 = 0; c4 < kInBlockScan / 4; ++c4) v[c4] = c4 < n4 ? q[c4] : make_int4(0, 0, 0, 0);
        int32_t all = 0, before = 0;
#pragma unroll
        for (int c4 = 0; c4 < kInBlockScan / 4; ++c4) {
          const int32_t x4[4] = {v[c4].x, v[c4].y, v[c4].z, v[c4].w};
#pragma unroll
          for (int q2 = 0; q2 < 4; ++q2) {
            all += x4[q2];
            before += 4 * c4 + q2 < chunk ? x4[q2] : 0;
          }
        }
        tot[e] = all;
        off[e] = before;
      }
    }
    __syncthreads();
    const int32_t total = block_excl_scan<TH>(tot, E, wtot);
    for (int e = tid; e < E; e += TH) off[e] += tot[e];
    if (chunk == 0) {
      const int eloc = E / a.N;
      for (int j = tid; j < a.N; j += TH) a.dest_off[j] = tot[j * eloc];
      if (tid == 0) a.dest_off[a.N] = total;
    }
  }
  __syncthreads();
  for (int e = tid; e < E; e += TH) {
    int32_t acc = off[e];
    for (int v = 0; v < kW; ++v) {
      const int32_t c = wc[v * E + e];
      wc[v * E + e] = acc;
      acc += c;
    }
  }
  __syncthreads();
  // every id's wave offset read first (clamped index), then the stores
  int at[kPT];
#pragma unroll
  for (int m = 0; m < kPT; ++m) at[m] = mine[(unsigned)ev[m] < (unsigned)E ? ev[m] : 0] + rk[m];
  uint8_t* const slot_out = a.sorted_slot;
#pragma unroll
  for (int m = 0; m < kPT; ++m) {
    if ((unsigned)ev[m] < (unsigned)E) {
      // x < 2^31 and k < 256: the multiply-high quotient is exact
      const uint32_t x = (uint32_t)(base + m * 64 + lane);
      const uint32_t t = (uint32_t)__umul64hi((uint64_t)x << 24, a.k_magic);
      a.sorted_tok[at[m]] = (int32_t)t;
      if (slot_out) slot_out[at[m]] = (uint8_t)(x - t * (uint32_t)a.k);
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

// Ids per histogram part: kThreads * 2^s with s in [2, 5].  Parts grow
// until a row has at most 16 of them (the merge then reads all of a row's
// parts in one round of loads), and beyond that while the launch still gets
// about 2,048 workgroups.
int64_t part_of(int32_t R, int64_t Tk) {
  int64_t part = (int64_t)kThreads * 4;
  while (part < (int64_t)kThreads * 32 &&
         ((Tk + part - 1) / part > 16 || (int64_t)R * ((Tk + 2 * part - 1) / (2 * part)) >= 2048))
    part *= 2;
  return part;
}

// Split of a call: ids per part, parts per row, sort chunks (and padded to 4).
struct DemandWs {
  int64_t part;
  int32_t P, nch, nch4;
};
DemandWs demand_ws(int32_t R, int64_t T, int32_t k) {
  DemandWs w;
  const int64_t Tk = T * k;
  w.part = part_of(R, Tk);
  w.P = (int32_t)std::max<int64_t>(1, (Tk + w.part - 1) / w.part);
  w.nch = std::max(1, n_chunks_of(Tk));
  w.nch4 = (w.nch + 3) / 4 * 4;
  return w;
}

}  // namespace

size_t demand_workspace(int32_t R, int64_t T, int32_t k, int32_t E) {
  const DemandWs w = demand_ws(R, T, k);
  const size_t partials = ((size_t)R * (size_t)w.P * (size_t)E * 4 + 255) / 256 * 256;
  return partials + (size_t)E * (size_t)w.nch4 * 4;
}

vp_status launch_demand(const DemandLaunch& a, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const int64_t Tk = a.T * a.k;
  const DemandWs w = demand_ws(a.R, a.T, a.k);
  const size_t partials = ((size_t)a.R * (size_t)w.P * (size_t)a.E * 4 + 255) / 256 * 256;
  char* ws = (char*)a.ws;
  int bits = 0;
  while ((1 << bits) < a.E) ++bits;
  const bool sorting = a.sort_row >= 0;
  const uint64_t k_magic = ((uint64_t(1) << 40) + (uint64_t)a.k - 1) / (uint64_t)a.k;
  DemandArgs d{a.routing, Tk, w.part, a.unit, a.E, a.N, a.first_rank, a.R, w.P, a.sort_row, w.nch, w.nch4, a.k,
               bits, k_magic, sorting && w.nch > kInBlockScan, a.counts, a.demand, a.sorted_tok, a.sorted_slot, a.dest_off,
               (int32_t*)ws, (int32_t*)(ws + partials), a.status};
  const int64_t blocks1 = (int64_t)a.R * w.P + (sorting ? w.nch : 0);
  if (blocks1 >= ((int64_t)1 << 31)) return set_error(VP_ERR_UNSUPPORTED, "too many histogram parts");
  hipLaunchKernelGGL(demand_count, dim3((unsigned)blocks1), dim3(kThreads), (size_t)kWaves * a.E * sizeof(int32_t),
                     s, d);
  if (d.scanned)
    hipLaunchKernelGGL(sort_scan, dim3(1), dim3(1024), 0, s, d.ccount, (int64_t)a.E * w.nch4, a.E, a.N, w.nch4,
                       a.dest_off);
  // pass 2: 512 threads when the chunk counts are held in registers (up to
  // 256 experts), else 256 (LDS: the chunk's offsets, totals and one count
  // row per wave)
  const int64_t blocks2 = (int64_t)a.R + (sorting ? w.nch : 0);
  const size_t lds256 = (size_t)(2 + 256 / 64) * a.E * sizeof(int32_t);
  const size_t lds512 = (size_t)(2 + 512 / 64) * a.E * sizeof(int32_t);
  if (d.scanned)
    hipLaunchKernelGGL((demand_finish<kOffScanned, 256>), dim3((unsigned)blocks2), dim3(256), lds256, s, d);
  else if (a.E <= 256)
    hipLaunchKernelGGL((demand_finish<kOffHeld, 512>), dim3((unsigned)blocks2), dim3(512), lds512, s, d);
  else
    hipLaunchKernelGGL((demand_finish<kOffReload, 256>), dim3((unsigned)blocks2), dim3(256), lds256, s, d);
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "demand launch failed");
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
