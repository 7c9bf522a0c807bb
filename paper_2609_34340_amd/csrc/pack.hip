// vp_pack: channel-ordered send buffers (Sec. 5 "Device-resident buffer
// layout").  For the steps in which this rank's lane carries bytes, in
// schedule order, the next x bytes of the stream to that step's destination
// are appended to the send buffer.
//
// Kernels
//   slices  one block: step offsets (exclusive scan of this rank's lane
//           volumes) and each step's offset inside its destination's stream
//           (a stable counting sort of the steps by destination -- ballot
//           match masks plus prefix popcounts -- followed by one scan).
//   index   one wavefront per step: the source byte offset of every packed
//           unit (a token row, or one head of one token).
//   gather  grid-stride 16-byte copy of the units into the send buffer with
//           non-temporal stores.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace vp {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ inline void report(int32_t* status, int code) { atomicCAS(status, 0, code); }

__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Exclusive block scan of v over 1024 threads; returns the exclusive prefix
// and writes the block total to *total.
__device__ int64_t block_excl_scan(int64_t v, int64_t* wsum, int64_t* total) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int64_t s = v;
  for (int o = 1; o < 64; o <<= 1) {
    int64_t y = __shfl_up(s, o);
    if (lane >= o) s += y;
  }
  if (lane == 63) wsum[w] = s;
  __syncthreads();
  int64_t before = 0, all = 0;
  for (int k = 0; k < 16; ++k) {
    if (k < w) before += wsum[k];
    all += wsum[k];
  }
  __syncthreads();
  *total = all;
  return before + s - v;
}

struct SliceArgs {
  int mode;
  const int32_t *Kp, *dst;
  const int64_t* bytes;
  int32_t k_max, N, self;
  int64_t unit, T, send_capacity, token_stride;
  const int64_t* dest_off;   // rows
  const int64_t* head_lo;    // heads
  int64_t* step_off;
  int64_t* cstream;          // per step: offset inside the destination stream (bytes)
  int32_t* status;
};

__global__ void __launch_bounds__(1024) slices_kernel(SliceArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int N = a.N, B = N + 1;   // bucket N collects the empty steps
  int64_t* xs = (int64_t*)smem;                       // k_max
  int64_t* xsum = xs + a.k_max;                       // B
  int64_t* base = xsum + B;                           // B
  int32_t* jv = (int32_t*)(base + B);                 // k_max
  int32_t* pos = jv + a.k_max;                        // k_max
  int32_t* cnt = pos + a.k_max;                       // B
  int32_t* run = cnt + B;                             // B
  __shared__ int64_t wsum[16];
  __shared__ int64_t carry, carry2;
  __shared__ int32_t Ks;

  if (tid == 0) {
    int K = *a.Kp;
    if (K < 0 || K > a.k_max) {
      report(a.status, VP_ERR_INVALID_ARGUMENT);
      K = 0;
    }
    // every head a destination owns must lie inside the token row
    if (a.mode == 1 && (a.head_lo[0] < 0 || a.head_lo[N] * a.unit > a.token_stride)) {
      report(a.status, VP_ERR_INVALID_ARGUMENT);
      K = 0;
    }
    Ks = K;
    carry = 0;
  }
  for (int b = tid; b < B; b += 1024) {
    cnt[b] = 0;
    xsum[b] = 0;
  }
  __syncthreads();
  const int K = Ks;
  // 1. lane volumes, validation, per-destination counts and sums, step offsets
  for (int k0 = 0; k0 < K; k0 += 1024) {
    const int k = k0 + tid;
    int64_t x = 0;
    if (k < K) {
      x = a.bytes[(size_t)k * N + a.self];
      const int j = a.dst[(size_t)k * N + a.self];
      int b = N;
      if (x != 0) {
        if (x < 0 || x % a.unit != 0 || j < 0 || j >= N || j == a.self) {
          report(a.status, VP_ERR_INVALID_ARGUMENT);
          x = 0;
        } else {
          b = j;
        }
      }
      jv[k] = b;
      atomicAdd(&cnt[b], 1);
      atomicAdd((unsigned long long*)&xsum[b], (unsigned long long)x);
    }
    int64_t tot;
    const int64_t e = block_excl_scan(x, wsum, &tot);
    if (k < K) a.step_off[k] = carry + e;
    __syncthreads();
    if (tid == 0) carry += tot;
    __syncthreads();
  }
  if (tid == 0) {
    a.step_off[K] = carry;
    if (carry > a.send_capacity) report(a.status, VP_ERR_CAPACITY);
  }
  __syncthreads();
  // 2. bucket starts (counts) and byte bases (sums)
  if (tid == 0) {
    carry = 0;
    carry2 = 0;
  }
  __syncthreads();
  for (int b0 = 0; b0 < B; b0 += 1024) {
    const int b = b0 + tid;
    const int64_t c = b < B ? cnt[b] : 0, xv = b < B ? xsum[b] : 0;
    int64_t tc, tx;
    const int64_t ec = block_excl_scan(c, wsum, &tc);
    const int64_t ex = block_excl_scan(xv, wsum, &tx);
    if (b < B) {
      run[b] = (int32_t)(carry + ec);
      base[b] = carry2 + ex;
    }
    __syncthreads();
    if (tid == 0) {
      carry += tc;
      carry2 += tx;
    }
    __syncthreads();
  }
  // 3. stable position of every step inside its destination bucket
  if (w == 0) {
    int bits = 0;
    while ((1 << bits) < B) ++bits;
    const uint64_t lt = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    for (int k0 = 0; k0 < K; k0 += 64) {
      const int k = k0 + lane;
      const bool live = k < K;
      const int b = live ? jv[k] : 0;
      uint64_t same = __ballot(live);
      for (int bt = 0; bt < bits; ++bt) {
        const uint64_t ones = __ballot(live && ((b >> bt) & 1));
        same &= ((b >> bt) & 1) ? ones : ~ones;
      }
      int p = 0;
      if (live) p = run[b] + __popcll(same & lt);
      wave_sync();
      if (live) {
        pos[k] = p;
        if ((same & lt) == 0) run[b] += __popcll(same);
      }
      wave_sync();
    }
  }
  __syncthreads();
  // 4. volumes in (destination, step) order, then one exclusive scan
  for (int k = tid; k < K; k += 1024) {
    int64_t x = jv[k] < N ? a.bytes[(size_t)k * N + a.self] : 0;
    xs[pos[k]] = x;
  }
  if (tid == 0) carry2 = 0;
  __syncthreads();
  for (int k0 = 0; k0 < K; k0 += 1024) {
    const int k = k0 + tid;
    const int64_t x = k < K ? xs[k] : 0;
    int64_t tot;
    const int64_t e = block_excl_scan(x, wsum, &tot);
    if (k < K) xs[k] = carry2 + e;
    __syncthreads();
    if (tid == 0) carry2 += tot;
    __syncthreads();
  }
  // 5. offset of each step inside its destination's stream; bounds check
  for (int k = tid; k < K; k += 1024) {
    const int b = jv[k];
    if (b == N) {
      a.cstream[k] = 0;
      continue;
    }
    const int64_t c = xs[pos[k]] - base[b];
    const int64_t x = a.bytes[(size_t)k * N + a.self];
    int64_t len;
    if (a.mode == 0) len = (a.dest_off[b + 1] - a.dest_off[b]) * a.unit;
    else len = a.T * (a.head_lo[b + 1] - a.head_lo[b]) * a.unit;
    if (c + x > len) report(a.status, VP_ERR_INVALID_ARGUMENT);
    a.cstream[k] = c;
  }
}

struct IndexArgs {
  int mode;
  const int32_t *Kp, *dst;
  const int64_t* bytes;
  int32_t N, self;
  int64_t unit, T, token_stride;
  const int32_t* sorted_tok;
  const int64_t* dest_off;
  const int64_t* head_lo;
  const int64_t* step_off;
  const int64_t* cstream;
  int64_t* src_off;
  int32_t* status;
};

__global__ void __launch_bounds__(64) index_kernel(IndexArgs a) {
  const int k = blockIdx.x, lane = threadIdx.x;
  if (k >= *a.Kp || *a.status != 0) return;
  const int64_t x = a.bytes[(size_t)k * a.N + a.self];
  if (x <= 0) return;
  const int j = a.dst[(size_t)k * a.N + a.self];
  const int64_t nu = x / a.unit, u0 = a.step_off[k] / a.unit, p0 = a.cstream[k] / a.unit;
  if (a.mode == 0) {
    const int64_t first = a.dest_off[j] + p0;
    for (int64_t u = lane; u < nu; u += 64) {
      const int64_t tok = a.sorted_tok[first + u];
      if (tok < 0 || tok >= a.T) {
        report(a.status, VP_ERR_INVALID_ARGUMENT);
        a.src_off[u0 + u] = 0;
      } else {
        a.src_off[u0 + u] = tok * a.unit;
      }
    }
  } else {
    const int64_t h0 = a.head_lo[j], h = a.head_lo[j + 1] - h0;
    for (int64_t u = lane; u < nu; u += 64) {
      const int64_t p = p0 + u, tok = p / h, hd = h0 + (p - tok * h);
      a.src_off[u0 + u] = tok * a.token_stride + hd * a.unit;
    }
  }
}

constexpr int kGatherThreads = 256;
constexpr int kGatherUnroll = 4;

__global__ void __launch_bounds__(kGatherThreads) gather_kernel(const unsigned char* __restrict__ src,
                                                                const int64_t* __restrict__ src_off,
                                                                const int32_t* Kp, const int64_t* step_off,
                                                                int64_t unit, int64_t vpu, uint64_t magic,
                                                                unsigned char* __restrict__ send,
                                                                const int32_t* status) {
  if (*status != 0) return;
  const int64_t total_vec = step_off[*Kp] / 16;
  const int64_t stride = (int64_t)gridDim.x * kGatherThreads;
  int64_t v = (int64_t)blockIdx.x * kGatherThreads + threadIdx.x;
  for (; v + (kGatherUnroll - 1) * stride < total_vec; v += kGatherUnroll * stride) {
    u32x4 r[kGatherUnroll];
#pragma unroll
    for (int m = 0; m < kGatherUnroll; ++m) {
      const uint64_t vv = (uint64_t)(v + m * stride);
      const int64_t u = (int64_t)__umul64hi(vv << 16, magic);
      const int64_t in = (int64_t)vv - u * vpu;
      r[m] = *(const u32x4*)(src + src_off[u] + in * 16);
    }
#pragma unroll
    for (int m = 0; m < kGatherUnroll; ++m)
      __builtin_nontemporal_store(r[m], (u32x4*)(send + (v + m * stride) * 16));
  }
  for (; v < total_vec; v += stride) {
    const int64_t u = (int64_t)__umul64hi((uint64_t)v << 16, magic);
    const int64_t in = v - u * vpu;
    u32x4 r = *(const u32x4*)(src + src_off[u] + in * 16);
    __builtin_nontemporal_store(r, (u32x4*)(send + v * 16));
  }
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace

size_t pack_workspace(int32_t k_max, int64_t send_capacity, int64_t unit) {
  size_t units = (size_t)(send_capacity / unit) + 1;
  return align_up((size_t)(k_max + 1) * sizeof(int64_t), 256) + units * sizeof(int64_t);
}

vp_status launch_pack(const PackLaunch& a, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const int B = a.N + 1;
  const size_t lds = (size_t)a.k_max * (8 + 4 + 4) + (size_t)B * (8 + 8 + 4 + 4);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return set_error(VP_ERR_HIP, "hipGetDevice failed");
  int lds_max = 0;
  if (hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
    return set_error(VP_ERR_HIP, "hipDeviceGetAttribute failed");
  if (lds + 1024 > (size_t)lds_max) return set_error(VP_ERR_UNSUPPORTED, "k_max too large for the slice table");
  if (a.unit % 16 != 0) return set_error(VP_ERR_INVALID_ARGUMENT, "unit must be a multiple of 16");
  int64_t* cstream = (int64_t*)a.ws;
  int64_t* src_off = (int64_t*)((char*)a.ws + align_up((size_t)(a.k_max + 1) * sizeof(int64_t), 256));

  if (a.stages & 1) {
    SliceArgs sa{a.mode, a.K, a.dst, a.bytes, a.k_max, a.N, a.self_rank, a.unit, a.T, a.send_capacity,
                 a.token_stride, a.dest_off, a.head_lo, a.step_off, cstream, a.status};
    if (hipFuncSetAttribute((const void*)slices_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
        hipSuccess)
      return set_error(VP_ERR_HIP, "cannot raise the slice kernel's LDS limit");
    hipLaunchKernelGGL(slices_kernel, dim3(1), dim3(1024), lds, s, sa);

    IndexArgs ia{a.mode, a.K, a.dst, a.bytes, a.N, a.self_rank, a.unit, a.T, a.token_stride, a.sorted_tok,
                 a.dest_off, a.head_lo, a.step_off, cstream, src_off, a.status};
    hipLaunchKernelGGL(index_kernel, dim3(a.k_max), dim3(64), 0, s, ia);
  }
  if (!(a.stages & 2)) {
    if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "pack launch failed");
    return VP_OK;
  }
  const int64_t vpu = a.unit / 16;
  // u = floor(v / vpu) = mulhi(v << 16, ceil(2^48 / vpu)) for v < 2^48 / vpu
  const unsigned __int128 two48 = (unsigned __int128)1 << 48;
  const uint64_t magic = (uint64_t)((two48 + (unsigned __int128)vpu - 1) / (unsigned __int128)vpu);
  const int64_t max_vec = a.send_capacity / 16;
  if (max_vec >= ((int64_t)1 << 48) / vpu) return set_error(VP_ERR_UNSUPPORTED, "send buffer too large");
  int64_t blocks = (max_vec + kGatherThreads * kGatherUnroll - 1) / (kGatherThreads * kGatherUnroll);
  blocks = std::max<int64_t>(1, std::min<int64_t>(blocks, 8192));
  hipLaunchKernelGGL(gather_kernel, dim3((unsigned)blocks), dim3(kGatherThreads), 0, s,
                     (const unsigned char*)a.src, src_off, a.K, a.step_off, a.unit, vpu, magic,
                     (unsigned char*)a.send, a.status);
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "pack launch failed");
  return VP_OK;
}

}  // namespace vp
