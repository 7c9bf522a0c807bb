// Receive side of the Sec. 5 buffer layout, and the combine direction.
//
// A receive buffer holds the slices addressed to one rank in step order, one
// token row per slot whose stride is the row rounded up to 128 bytes (Sec. 5
// low-latency protocol: every row starts 128-byte aligned).  The dispatch
// receive is unpacked into the expert-major output: local expert m's rows from
// source 0, then source 1, ..., each source's rows in token order, which is
// the order of the stream from that source (Sec. 5: the receive kernel writes
// the output layout directly).  The combine returns every row to its source
// rank with a schedule planned on the transposed demand (the return AlltoAllv
// of expert parallelism); its pack reads the expert-major rows in stream
// order and its unpack puts every returned row at (token, routing slot).
//
// Kernels
//   map    one workgroup per step.  It takes the lane that moves rows to (or
//          from) this rank at its step, sums the volumes of this rank's
//          earlier steps (where the slice sits in the receive or send buffer)
//          and of its earlier steps with the same peer (where it sits in that
//          stream), and writes, for every row of the slice, the row index on
//          the other side: an expert-major output row, or token * k + slot.
//          The workgroup of the last step also checks that every peer's
//          stream is covered exactly.
//   copy   one workgroup per buffer row, each XCD a contiguous eighth of
//          the rows: 16-byte loads issued a pass at a time ahead of the
//          non-temporal stores.
//   transpose  D^T for the combine's plan, in 32 x 32 LDS tiles.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"

namespace vp {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

__device__ inline void report(int32_t* status, int code) { atomicCAS(status, 0, code); }

constexpr int kMapThreads = 256;
constexpr int kMapWaves = kMapThreads / 64;

struct MapArgs {
  int mode, self, N, k_max, eloc, E, k;
  int64_t rb, T;
  int64_t rows_cap;   // rows the buffer side holds (receive slots, or send rows)
  int64_t map_cap;    // rows the other side holds (expert-major output, or T * k)
  const int32_t *Kp, *dst, *recv_src;
  const int64_t* bytes;
  const int32_t* counts;        // [N][E] dispatch assignments per (source rank, expert)
  const int32_t* sorted_tok;
  const uint8_t* sorted_slot;
  const int64_t* dest_off;
  int64_t* step_off;            // pack combine: [k_max + 1]
  int32_t* map;                 // [rows_cap]
  int64_t* total;               // rows in the buffer
  int32_t* status;
};

// Sum over the block; every thread gets it.
__device__ int64_t block_sum(int64_t v, int64_t* red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  int64_t s = 0;
  for (int i = 0; i < kMapWaves; ++i) s += red[i];
  return s;
}

// Exclusive scan of v[0, n) in LDS by the whole block; returns the total.
__device__ int64_t block_excl_scan(int64_t* v, int n, int64_t* red) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int per = (n + kMapThreads - 1) / kMapThreads;
  const int b = min(tid * per, n), e = min(b + per, n);
  int64_t s = 0;
  for (int i = b; i < e; ++i) s += v[i];
  int64_t incl = s;
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  __syncthreads();
  if (lane == 63) red[w] = incl;
  __syncthreads();
  int64_t run = incl - s, total = 0;
  for (int i = 0; i < kMapWaves; ++i) {
    if (i < w) run += red[i];
    total += red[i];
  }
  for (int i = b; i < e; ++i) {
    const int64_t t = v[i];
    v[i] = run;
    run += t;
  }
  __syncthreads();
  return total;
}

__global__ void __launch_bounds__(kMapThreads) map_kernel(MapArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ int64_t red[kMapWaves];
  __shared__ int32_t sK, sst;
  const int k = blockIdx.x, tid = threadIdx.x, N = a.N, self = a.self;
  if (tid == 0) {   // one read, so that every early exit below is taken by the whole block
    sK = *a.Kp;
    sst = *a.status;
  }
  __syncthreads();
  const int K = sK;
  if (K < 0 || K > a.k_max) {
    if (k == 0 && tid == 0) report(a.status, VP_ERR_INVALID_ARGUMENT);
    return;
  }
  if (sst != 0) return;
  if (k >= K) {
    if (k == 0 && tid == 0) {   // an empty schedule moves nothing
      *a.total = 0;
      if (a.step_off) a.step_off[0] = 0;
    }
    return;
  }
  const bool recv = a.mode != kModeCombinePack;

  // 1. this step: the lane carrying rows to or from this rank, and its peer
  int lane_k, peer;
  bool ok;
  if (recv) {
    lane_k = a.recv_src[(size_t)k * N + self];
    ok = lane_k >= 0 && lane_k < N && a.dst[(size_t)k * N + lane_k] == self;
    peer = lane_k;
  } else {
    lane_k = self;
    peer = a.dst[(size_t)k * N + self];
    ok = peer >= 0 && peer < N;
  }
  const int64_t x = ok ? a.bytes[(size_t)k * N + lane_k] : 0;
  ok = ok && x >= 0 && x % a.rb == 0 && (x == 0 || peer != self);
  if (!ok) {
    if (tid == 0) report(a.status, VP_ERR_INVALID_ARGUMENT);
    return;
  }

  // 2. volumes of this rank's earlier steps, in total and with the same peer;
  //    the last step's workgroup also counts every peer's rows
  const bool last = k == K - 1;
  int64_t* tot = (int64_t*)smem;   // [N] rows per peer (last step only)
  if (last)
    for (int j = tid; j < N; j += kMapThreads) tot[j] = 0;
  __syncthreads();
  int64_t pos = 0, strm = 0;
  const int kend = last ? K : k;
  for (int kk = tid; kk < kend; kk += kMapThreads) {
    int s = self, p;
    if (recv) {
      s = a.recv_src[(size_t)kk * N + self];
      p = s;
    } else {
      p = a.dst[(size_t)kk * N + self];
    }
    // a lane that does not match the schedule is reported by its step's own
    // workgroup and left out here
    if (s < 0 || s >= N || p < 0 || p >= N || (recv && a.dst[(size_t)kk * N + s] != self)) continue;
    const int64_t xx = a.bytes[(size_t)kk * N + s];
    if (kk < k) {
      pos += xx;
      if (p == peer) strm += xx;
    }
    if (last && xx > 0) atomicAdd((unsigned long long*)&tot[p], (unsigned long long)(xx / a.rb));
  }
  pos = block_sum(pos, red);
  strm = block_sum(strm, red);
  const int64_t g0 = pos / a.rb, nu = x / a.rb, q0 = strm / a.rb;
  if (tid == 0) {
    if (a.step_off) a.step_off[k] = pos;
    if (last) {
      *a.total = g0 + nu;
      if (a.step_off) a.step_off[K] = pos + x;
    }
  }
  if (pos < 0 || strm < 0 || g0 + nu > a.rows_cap) {
    if (tid == 0) report(a.status, pos < 0 || strm < 0 ? VP_ERR_INVALID_ARGUMENT : VP_ERR_CAPACITY);
    return;
  }

  // 3. last step: every peer's stream must be delivered whole -- the rows of
  //    the peer's assignments to this rank's experts (dispatch receive, and the
  //    same rows sent back by the combine), or this rank's rows for that peer
  //    (combine receive)
  if (last) {
    if (a.mode == kModeCombineUnpack) {
      for (int p = tid; p < N; p += kMapThreads)
        if (p != self)
          atomicAdd((unsigned long long*)&tot[p], (unsigned long long)-(a.dest_off[p + 1] - a.dest_off[p]));
    } else {
      const int n = N * a.eloc;
      for (int idx = tid; idx < n; idx += kMapThreads) {
        const int p = idx / a.eloc, m = idx - p * a.eloc;
        if (p != self)
          atomicAdd((unsigned long long*)&tot[p],
                    (unsigned long long)-(int64_t)a.counts[(size_t)p * a.E + (size_t)self * a.eloc + m]);
      }
    }
    __syncthreads();
    for (int p = tid; p < N; p += kMapThreads)
      if (tot[p] != 0) report(a.status, VP_ERR_INVALID_ARGUMENT);
  }
  if (nu == 0) return;

  // 4. the row on the other side of every row of this slice
  if (a.mode == kModeCombineUnpack) {
    const int64_t b0 = a.dest_off[peer], len = a.dest_off[peer + 1] - b0;
    if (b0 < 0 || len < 0 || b0 + len > a.map_cap || q0 + nu > len) {   // sorted lists hold T * k entries
      if (tid == 0) report(a.status, VP_ERR_INVALID_ARGUMENT);
      return;
    }
    for (int64_t u = tid; u < nu; u += kMapThreads) {
      const int64_t p = b0 + q0 + u;
      const int64_t t = a.sorted_tok[p];
      const int c = a.sorted_slot[p];
      if (t < 0 || t >= a.T || c >= a.k) {
        report(a.status, VP_ERR_INVALID_ARGUMENT);
        continue;
      }
      a.map[g0 + u] = (int32_t)(t * a.k + c);
    }
    return;
  }
  // expert-major output: expert m's rows start at base[m] = rows of experts
  // before m from every source + rows of m from sources before the peer; the
  // peer's stream holds its rows for expert m from cum[m] on
  const int eloc = a.eloc;
  int64_t* base = (int64_t*)smem + N;   // [eloc]
  int64_t* part = base + eloc;          // [eloc]
  int64_t* cum = part + eloc;           // [eloc + 1]
  for (int m = tid; m < eloc; m += kMapThreads) {
    base[m] = 0;
    part[m] = 0;
    cum[m] = a.counts[(size_t)peer * a.E + (size_t)self * eloc + m];
  }
  __syncthreads();
  const int n = N * eloc;
  for (int idx = tid; idx < n; idx += kMapThreads) {
    const int i = idx / eloc, m = idx - i * eloc;
    const int64_t c = a.counts[(size_t)i * a.E + (size_t)self * eloc + m];
    atomicAdd((unsigned long long*)&base[m], (unsigned long long)c);
    if (i < peer) atomicAdd((unsigned long long*)&part[m], (unsigned long long)c);
  }
  __syncthreads();
  const int64_t out_rows = block_excl_scan(base, eloc, red);
  const int64_t stream_rows = block_excl_scan(cum, eloc, red);
  if (q0 + nu > stream_rows || out_rows > a.map_cap) {
    if (tid == 0) report(a.status, q0 + nu > stream_rows ? VP_ERR_INVALID_ARGUMENT : VP_ERR_CAPACITY);
    return;
  }
  for (int64_t u = tid; u < nu; u += kMapThreads) {
    const int64_t q = q0 + u;
    int lo = 0, hi = eloc - 1;   // the last expert whose rows start at or before q
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (cum[mid] <= q) lo = mid;
      else hi = mid - 1;
    }
    const int64_t row = base[lo] + part[lo] + (q - cum[lo]);
    if (row < 0 || row >= a.map_cap) {
      report(a.status, VP_ERR_INVALID_ARGUMENT);
      continue;
    }
    a.map[g0 + u] = (int32_t)row;
  }
}

// Buffer row g <-> mapped row map[g]: read from the mapped side (map_src) or
// write to it.  Rows are whole 16-byte vectors.  One workgroup per row; TH
// threads move it in passes of V vectors per thread, every load of a pass
// issued before its stores (about 2 KiB in flight per wavefront, as for the
// dispatch scatter).
template <int TH, int V>
__global__ void __launch_bounds__(TH) copy_rows_kernel(const unsigned char* __restrict__ src, int64_t src_stride,
                                                       unsigned char* __restrict__ dst, int64_t dst_stride,
                                                       int64_t vpr, const int32_t* __restrict__ map, int map_src,
                                                       const int64_t* total, int64_t rows_cap,
                                                       const int32_t* status) {
  if (*status != 0) return;
  int64_t U = *total;
  U = U < rows_cap ? U : rows_cap;
  // XCD x (block % 8) copies the x-th eighth of the buffer's rows, in order
  // (measured 4-6 % faster than rows dealt to the XCDs in turn); the grid
  // covers rows_cap rounded up to eight, and blocks past the rows exit
  const int64_t per = (U + 7) / 8;
  const int64_t j = blockIdx.x >> 3;
  if (j >= per) return;
  const int64_t g = (int64_t)(blockIdx.x & 7) * per + j;
  if (g >= U) return;
  const int64_t m = map[g];
  const int64_t sr = map_src ? m : g, dr = map_src ? g : m;
  const u32x4* s = (const u32x4*)(src + sr * src_stride);
  u32x4* d = (u32x4*)(dst + dr * dst_stride);
  for (int64_t e0 = threadIdx.x; e0 < vpr; e0 += (int64_t)V * TH) {
    u32x4 r[V];
#pragma unroll
    for (int i = 0; i < V; ++i)
      if (e0 + i * TH < vpr) r[i] = s[e0 + i * TH];
#pragma unroll
    for (int i = 0; i < V; ++i)
      if (e0 + i * TH < vpr) __builtin_nontemporal_store(r[i], d + e0 + i * TH);
  }
}

constexpr int kTile = 32;

__global__ void __launch_bounds__(kTile * 8) transpose_kernel(const int64_t* __restrict__ D, int N,
                                                              int64_t* __restrict__ DT) {
  __shared__ int64_t tile[kTile][kTile + 1];
  const int bx = blockIdx.x * kTile, by = blockIdx.y * kTile;
  const int tx = threadIdx.x & (kTile - 1), ty = threadIdx.x / kTile;
  for (int r = ty; r < kTile; r += 8) {
    const int i = by + r, j = bx + tx;
    if (i < N && j < N) tile[r][tx] = D[(size_t)i * N + j];
  }
  __syncthreads();
  for (int r = ty; r < kTile; r += 8) {
    const int j = bx + r, i = by + tx;
    if (i < N && j < N) DT[(size_t)j * N + i] = tile[tx][r];
  }
}

constexpr size_t kHeader = 256;   // [0]: rows in the buffer (int64)

}  // namespace

int64_t slot_bytes(int64_t row_bytes) { return (row_bytes + 127) / 128 * 128; }

size_t unpack_workspace(int64_t rows) { return kHeader + align_up((size_t)rows * 4, 256); }

size_t unpack_lds_bytes(int mode, int32_t N, int32_t eloc) {
  return (size_t)N * 8 + (mode == kModeCombineUnpack ? 0 : (size_t)(3 * eloc + 1) * 8);
}

vp_status launch_unpack(const UnpackLaunch& a, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const int eloc = a.E / a.N;
  const size_t lds = unpack_lds_bytes(a.mode, a.N, eloc);
  if (lds > 64 * 1024) return set_error(VP_ERR_UNSUPPORTED, "too many ranks or local experts for the row map");
  char* ws = (char*)a.ws;
  int64_t* total = (int64_t*)ws;
  int32_t* map = (int32_t*)(ws + kHeader);
  MapArgs m{a.mode, a.self_rank, a.N, a.k_max, eloc, a.E, a.k, a.row_bytes, a.T, a.rows_cap, a.map_cap,
            a.K, a.dst, a.recv_src, a.bytes, a.counts, a.sorted_tok, a.sorted_slot, a.dest_off, a.step_off,
            map, total, a.status};
  hipLaunchKernelGGL(map_kernel, dim3(a.k_max), dim3(kMapThreads), lds, s, m);
  if (a.rows_cap > 0) {
    if (a.rows_cap >= ((int64_t)1 << 31) - 8) return set_error(VP_ERR_UNSUPPORTED, "too many buffer rows");
    const int64_t vpr = a.row_bytes / 16;
    const dim3 grid((unsigned)((a.rows_cap + 7) / 8 * 8));   // rows past the buffer's count exit at once
    const unsigned char* sp = (const unsigned char*)a.src;
    unsigned char* dp = (unsigned char*)a.dst_buf;
    const int ms = a.mode == kModeCombinePack ? 1 : 0;
    // about 2 KiB per wavefront: rows up to 2, 4 and 8 KiB take 1, 2 and 4
    // wavefronts of two vectors per thread, longer rows 8 wavefronts of one
    if (vpr <= 128)
      hipLaunchKernelGGL((copy_rows_kernel<64, 2>), grid, dim3(64), 0, s, sp, a.src_stride, dp, a.dst_stride, vpr,
                         map, ms, total, a.rows_cap, a.status);
    else if (vpr <= 256)
      hipLaunchKernelGGL((copy_rows_kernel<128, 2>), grid, dim3(128), 0, s, sp, a.src_stride, dp, a.dst_stride, vpr,
                         map, ms, total, a.rows_cap, a.status);
    else if (vpr <= 512)
      hipLaunchKernelGGL((copy_rows_kernel<256, 2>), grid, dim3(256), 0, s, sp, a.src_stride, dp, a.dst_stride, vpr,
                         map, ms, total, a.rows_cap, a.status);
    else
      hipLaunchKernelGGL((copy_rows_kernel<512, 1>), grid, dim3(512), 0, s, sp, a.src_stride, dp, a.dst_stride, vpr,
                         map, ms, total, a.rows_cap, a.status);
  }
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "unpack launch failed");
  return VP_OK;
}

vp_status launch_transpose(const int64_t* D, int32_t N, int64_t* DT, void* stream) {
  const unsigned b = (unsigned)((N + kTile - 1) / kTile);
  hipLaunchKernelGGL(transpose_kernel, dim3(b, b), dim3(kTile * 8), 0, (hipStream_t)stream, D, N, DT);
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "transpose launch failed");
  return VP_OK;
}

}  // namespace vp
