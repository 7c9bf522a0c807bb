// vp_plan: online channel-guided demand decomposition (Sec. 4.2, Alg. 2) as
// one persistent workgroup of 1024 threads that runs the whole iteration
// loop on the device.
//
// Per iteration:
//   1. shape scores, Eq. (5)-(6), from node-block aggregates kept in LDS:
//      A = sum over nodes of the diagonal node block of D-hat and B_k = sum of
//      the blocks (n, n+k).  A shape (k, L, R) scores sum A.L + sum B_k.R,
//      which equals sum D-hat.M (the aggregates are updated incrementally by
//      each activation's lanes, so D-hat itself is never materialised);
//      argmax with ties to the lowest shape index via one packed 64-bit key;
//   2. for the families of the best shape: the binding credits
//      h' = min(D^rem_ij, cap) (Eq. (7) scaled by tau) of every instance and
//      endpoint pair are gathered into LDS once;
//   3. MultiStartAA (Eq. (8)): one wavefront per (family, start) builds the
//      start, runs the alternating source / destination halves (all groups of
//      a half in parallel across lanes) and reports F and the slowest lane;
//   4. Evaluate (Eq. (9)-(10)) and the exact utility argmax in 128-bit;
//   5. the activation is appended and subtracted from D^rem (global, L2
//      resident) and from the aggregates.
// No host round trip happens between iterations.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"

namespace vp {
namespace {

constexpr int kWaves = kPlanThreads / 64;
constexpr int kMaxQG = kMaxSlotsPerNode * kMaxGpusPerSwitch;   // lanes per node
constexpr int kMaxPerm = 24;                                   // 4!

struct PairRes {
  int64_t F;
  int64_t xmax[3];
};

struct ChunkFam {
  int32_t f, k;
  int32_t info[kMaxQG];      // cls | src_slot<<4 | dst_slot<<8 | local_id<<12
  uint8_t outl[kMaxQG];      // [slot][m] local index
  uint8_t inl[kMaxQG];
};

struct Shared {
  uint64_t key;
  int64_t total_rem, S, Lmax, tau;
  int64_t cap[3];
  int64_t best_S, best_xm, best_bm;
  int32_t K, err, best_valid, best_f, best_k, copy_pair;
  int32_t fam_begin, fam_end;
  int64_t red[kWaves + 1];
  uint8_t perms[kMaxPerm * kMaxGpusPerSwitch];
};

struct PlanArgs {
  const int32_t* cat;
  DevCatalogLayout L;
  const int64_t* D;
  int64_t* Drem;
  int64_t k_target, lambda, unit;
  uint64_t seed;
  uint64_t odd_inv, odd_lim;
  int32_t unit_shift;
  int32_t n_start, i_aa, k_max, FC;
  int32_t *K, *family, *dst, *inst;
  int64_t *bytes, *tau;
  int32_t* status;
  int32_t o_rinfo, o_agg, o_terms, o_nterms, o_base, o_cf, o_pair, o_best, o_sh, o_hp, o_sl, o_dl;
};

// ------------------------------------------------------------------ helpers

__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ inline int64_t wave_sum(int64_t v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ inline int64_t wave_max(int64_t v) {
  for (int o = 32; o > 0; o >>= 1) v = max(v, (int64_t)__shfl_xor(v, o));
  return v;
}
__device__ inline uint64_t wave_max_u(uint64_t v) {
  for (int o = 32; o > 0; o >>= 1) {
    uint64_t w = __shfl_xor(v, o);
    v = w > v ? w : v;
  }
  return v;
}

// SplitMix64 (Steele, Lea, Flood 2014): key absorbs the fields one at a time.
constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
__device__ inline uint64_t sm_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Utility order of Eq. (10): (S1, x1/b1) beats (S2, x2/b2) exactly.
__device__ inline bool utility_greater(int64_t S1, int64_t x1, int64_t b1, int64_t S2, int64_t x2,
                                       int64_t b2, int64_t lam) {
  if (S1 == 0) return false;
  if (S2 == 0) return true;
  typedef unsigned __int128 u128;
  u128 lhs = (u128)S1 * (u128)b1 * ((u128)lam * (u128)b2 + (u128)x2);
  u128 rhs = (u128)S2 * (u128)b2 * ((u128)lam * (u128)b1 + (u128)x1);
  return lhs > rhs;
}

struct Fam {
  const ChunkFam* cf;
  const int32_t* rinfo;   // rank -> node<<8 | slot<<4 | local
  int Q, g, QG, nn, k;
  __device__ int node_of(int t) const { return rinfo[t] >> 8; }
  __device__ int src_group(int t) const {
    int n = node_of(t);
    return n * Q + ((cf->info[t - n * QG] >> 4) & 15);
  }
  __device__ int dst_group(int t) const {
    int n = node_of(t);
    int info = cf->info[t - n * QG];
    int dn = ((info & 15) == VP_PATH_NIC && k) ? (n + k) % nn : n;
    return dn * Q + ((info >> 8) & 15);
  }
  __device__ int cls(int t) const { return cf->info[t - node_of(t) * QG] & 15; }
  // the m-th out-instance of group a (family order)
  __device__ int out_t(int a, int m) const {
    int n = a / Q, q = a - n * Q;
    return n * QG + cf->outl[q * g + m];
  }
  // the in-instances of group d in family order (ascending instance index)
  __device__ void in_list(int d, int* tl) const {
    int n = d / Q, q = d - n * Q;
    for (int m = 0; m < g; ++m) {
      int idx = cf->inl[q * g + m];
      int c = cf->info[idx] & 15;
      int sn = (c == VP_PATH_NIC && k) ? (n - k + nn) % nn : n;
      tl[m] = sn * QG + idx;
    }
    for (int m = 1; m < g; ++m)
      for (int x = m; x > 0 && tl[x - 1] > tl[x]; --x) {
        int t = tl[x];
        tl[x] = tl[x - 1];
        tl[x - 1] = t;
      }
  }
};

// Self-binding repair: per group, each self-bound intra-group instance (in
// out-list order) trades destinations with the first other unprotected
// in-instance of the group, else sources with the first other unprotected
// out-instance.
__device__ void repair(const Fam& fm, uint8_t* SL, uint8_t* DL, int G, int protect, int lane) {
  const int g = fm.g;
  for (int a = lane; a < G; a += 64) {
    int o[kMaxGpusPerSwitch], tl[kMaxGpusPerSwitch];
    for (int m = 0; m < g; ++m) o[m] = fm.out_t(a, m);
    fm.in_list(a, tl);
    for (int m = 0; m < g; ++m) {
      int r = o[m];
      if (fm.dst_group(r) != a || SL[r] != DL[r]) continue;
      int partner = -1;
      for (int m2 = 0; m2 < g && partner < 0; ++m2)
        if (tl[m2] != r && tl[m2] != protect) partner = tl[m2];
      if (partner >= 0) {
        uint8_t x = DL[r];
        DL[r] = DL[partner];
        DL[partner] = x;
        continue;
      }
      for (int m3 = 0; m3 < g && partner < 0; ++m3)
        if (o[m3] != r && o[m3] != protect) partner = o[m3];
      if (partner >= 0) {
        uint8_t x = SL[r];
        SL[r] = SL[partner];
        SL[partner] = x;
      }
    }
  }
  wave_sync();
}

// One (family, start) pair: build the start, run AA, report F and the
// largest lane volume per path class.  Executed by one whole wavefront.
__device__ void run_pair(const PlanArgs& P, const Fam& fm, const uint32_t* H, uint8_t* SL, uint8_t* DL,
                         const Shared* sh, int start, int iter, int lane, PairRes* out) {
  const int g = fm.g, G = P.L.G, N = P.L.N, g2 = g * g;
  if (start == 0) {
    // canonical binding
    for (int a = lane; a < G; a += 64) {
      int tl[kMaxGpusPerSwitch];
      for (int m = 0; m < g; ++m) SL[fm.out_t(a, m)] = (uint8_t)m;
      fm.in_list(a, tl);
      for (int m = 0; m < g; ++m) DL[tl[m]] = (uint8_t)m;
    }
    wave_sync();
    // highest-credit triple, ties to the smallest (t, i, j)
    uint64_t best = 0;
    for (int t = lane; t < N; t += 64)
      for (int e = 0; e < g2; ++e) {
        uint32_t h = H[t * g2 + e];
        if (h != kForbidden && h > 0) {
          uint64_t key = ((uint64_t)h << 24) | (uint64_t)(0xFFFFFF - (t * g2 + e));
          best = key > best ? key : best;
        }
      }
    best = wave_max_u(best);
    int protect = -1;
    if (best) {
      int idx = 0xFFFFFF - (int)(best & 0xFFFFFF);
      int ts = idx / g2, e = idx - ts * g2;
      int il = e / g, jl = e - il * g;
      protect = ts;
      if (lane == 0) {
        int a = fm.src_group(ts);
        for (int m = 0; m < g; ++m) {
          int t2 = fm.out_t(a, m);
          if (SL[t2] == il) {
            SL[t2] = SL[ts];
            SL[ts] = (uint8_t)il;
            break;
          }
        }
        int tl[kMaxGpusPerSwitch];
        fm.in_list(fm.dst_group(ts), tl);
        for (int m = 0; m < g; ++m) {
          int t3 = tl[m];
          if (DL[t3] == jl) {
            DL[t3] = DL[ts];
            DL[ts] = (uint8_t)jl;
            break;
          }
        }
      }
      wave_sync();
    }
    repair(fm, SL, DL, G, protect, lane);
  } else {
    // independent Fisher-Yates shuffles of every group's sources and destinations
    for (int a = lane; a < G; a += 64) {
      for (int side = 0; side < 2; ++side) {
        uint64_t key = P.seed;
        key = sm_mix(key + kGolden) ^ (uint64_t)iter;
        key = sm_mix(key + kGolden) ^ (uint64_t)fm.cf->f;
        key = sm_mix(key + kGolden) ^ (uint64_t)start;
        key = sm_mix(key + kGolden) ^ (uint64_t)a;
        key = sm_mix(key + kGolden) ^ (uint64_t)side;
        uint64_t state = key;
        int perm[kMaxGpusPerSwitch];
        for (int m = 0; m < g; ++m) perm[m] = m;
        for (int m = g - 1; m >= 1; --m) {
          state += kGolden;
          int j = (int)(sm_mix(state) % (uint64_t)(m + 1));
          int x = perm[m];
          perm[m] = perm[j];
          perm[j] = x;
        }
        if (side == 0) {
          for (int m = 0; m < g; ++m) SL[fm.out_t(a, m)] = (uint8_t)perm[m];
        } else {
          int tl[kMaxGpusPerSwitch];
          fm.in_list(a, tl);
          for (int m = 0; m < g; ++m) DL[tl[m]] = (uint8_t)perm[m];
        }
      }
    }
    wave_sync();
    repair(fm, SL, DL, G, -1, lane);
  }

  // Alternating Algorithm: source half, then destination half.
  const int np = P.L.n_perm;
  const uint8_t* perms = sh->perms;
  for (int sweep = 0; sweep < P.i_aa; ++sweep) {
    int changed = 0;
    for (int a = lane; a < G; a += 64) {
      int o[kMaxGpusPerSwitch], jl[kMaxGpusPerSwitch];
      int64_t cur = 0;
      for (int m = 0; m < g; ++m) {
        o[m] = fm.out_t(a, m);
        jl[m] = DL[o[m]];
        cur += H[o[m] * g2 + SL[o[m]] * g + jl[m]];
      }
      int64_t bestv = -1;
      int bp = -1;
      for (int p = 0; p < np; ++p) {
        int64_t v = 0;
        bool ok = true;
        for (int m = 0; m < g; ++m) {
          uint32_t h = H[o[m] * g2 + perms[p * g + m] * g + jl[m]];
          if (h == kForbidden) { ok = false; break; }
          v += h;
        }
        if (ok && v > bestv) { bestv = v; bp = p; }
      }
      if (bestv > cur) {
        for (int m = 0; m < g; ++m) SL[o[m]] = perms[bp * g + m];
        changed = 1;
      }
    }
    wave_sync();
    for (int d = lane; d < G; d += 64) {
      int tl[kMaxGpusPerSwitch], il[kMaxGpusPerSwitch];
      fm.in_list(d, tl);
      int64_t cur = 0;
      for (int m = 0; m < g; ++m) {
        il[m] = SL[tl[m]];
        cur += H[tl[m] * g2 + il[m] * g + DL[tl[m]]];
      }
      int64_t bestv = -1;
      int bp = -1;
      for (int p = 0; p < np; ++p) {
        int64_t v = 0;
        bool ok = true;
        for (int m = 0; m < g; ++m) {
          uint32_t h = H[tl[m] * g2 + il[m] * g + perms[p * g + m]];
          if (h == kForbidden) { ok = false; break; }
          v += h;
        }
        if (ok && v > bestv) { bestv = v; bp = p; }
      }
      if (bestv > cur) {
        for (int m = 0; m < g; ++m) DL[tl[m]] = perms[bp * g + m];
        changed = 1;
      }
    }
    wave_sync();
    if (!__any(changed)) break;
  }

  // binding score F (Eq. (8)) and the largest lane volume per path class
  int64_t F = 0, x0 = 0, x1 = 0, x2 = 0;
  for (int t = lane; t < N; t += 64) {
    int64_t h = H[t * g2 + SL[t] * g + DL[t]];
    F += h;
    int c = fm.cls(t);
    if (c == 0) x0 = max(x0, h);
    else if (c == 1) x1 = max(x1, h);
    else x2 = max(x2, h);
  }
  F = wave_sum(F);
  x0 = wave_max(x0);
  x1 = wave_max(x1);
  x2 = wave_max(x2);
  if (lane == 0) {
    out->F = F;
    out->xmax[0] = x0;
    out->xmax[1] = x1;
    out->xmax[2] = x2;
  }
}

__device__ inline void set_err(Shared* sh, int code) { atomicCAS(&sh->err, 0, code); }

__global__ void __launch_bounds__(kPlanThreads) plan_kernel(PlanArgs P) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const DevCatalogLayout& L = P.L;
  const int N = L.N, g = L.g, Q = L.Q, nn = L.nn, QG = Q * g, g2 = g * g;
  const int NP = L.J0 + L.J1, NS = P.n_start;
  int32_t* rinfo = (int32_t*)(smem + P.o_rinfo);
  int64_t* agg = (int64_t*)(smem + P.o_agg);
  uint16_t* terms = (uint16_t*)(smem + P.o_terms);
  uint8_t* nterms = smem + P.o_nterms;
  int64_t* base = (int64_t*)(smem + P.o_base);
  ChunkFam* cf = (ChunkFam*)(smem + P.o_cf);
  PairRes* pr = (PairRes*)(smem + P.o_pair);
  uint8_t* bsl = smem + P.o_best;
  uint8_t* bdl = bsl + N;
  Shared* sh = (Shared*)(smem + P.o_sh);
  uint32_t* hp = (uint32_t*)(smem + P.o_hp);
  uint8_t* sl = smem + P.o_sl;
  uint8_t* dl = smem + P.o_dl;
  const int32_t* cat = P.cat;

  // ---------------------------------------------------------------- prologue
  if (tid == 0) {
    sh->err = 0;
    sh->K = 0;
    sh->total_rem = 0;
    sh->Lmax = 0;
  }
  for (int x = tid; x < L.n_perm * g; x += kPlanThreads) sh->perms[x] = (uint8_t)cat[L.off_perms + x];
  for (int r = tid; r < N; r += kPlanThreads) {
    int grp = r / g;
    rinfo[r] = ((grp / Q) << 8) | ((grp % Q) << 4) | (r - grp * g);
  }
  for (int x = tid; x < NP * L.TS; x += kPlanThreads) terms[x] = (uint16_t)cat[L.off_terms + x];
  for (int p = tid; p < NP; p += kPlanThreads) nterms[p] = (uint8_t)cat[L.off_nterms + p];
  for (int x = tid; x < nn * Q * Q; x += kPlanThreads) agg[x] = 0;
  int64_t* colsum = (int64_t*)hp;   // the credit area is free during the prologue
  for (int x = tid; x < N; x += kPlanThreads) colsum[x] = 0;
  __syncthreads();

  // one pass over D: validate, copy to D^rem, row / column sums, aggregates
  {
    bool bad = false;
    int64_t tot = 0, lmax = 0;
    const uint64_t mask = (uint64_t(1) << P.unit_shift) - 1;
    for (int i = wave; i < N; i += kWaves) {
      const int ri = rinfo[i], ni = ri >> 8, qi = (ri >> 4) & 15;
      int64_t rs = 0;
      for (int j = lane; j < N; j += 64) {
        int64_t v = P.D[(size_t)i * N + j];
        bool divisible = ((uint64_t)v & mask) == 0 &&
                         ((uint64_t)v >> P.unit_shift) * P.odd_inv <= P.odd_lim;
        if (v < 0 || (i == j && v != 0) || !divisible) bad = true;
        P.Drem[(size_t)i * N + j] = v;
        rs += v;
        if (v > 0) {
          const int rj = rinfo[j], nj = rj >> 8, qj = (rj >> 4) & 15;
          int kk = nj - ni;
          if (kk < 0) kk += nn;
          atomicAdd((unsigned long long*)&colsum[j], (unsigned long long)v);
          atomicAdd((unsigned long long*)&agg[(kk * Q + qi) * Q + qj], (unsigned long long)v);
        }
      }
      rs = wave_sum(rs);
      tot += rs;
      lmax = max(lmax, rs);
    }
    if (bad) set_err(sh, VP_ERR_INVALID_DEMAND);
    if (lane == 0) {
      atomicAdd((unsigned long long*)&sh->total_rem, (unsigned long long)tot);
      atomicMax((unsigned long long*)&sh->Lmax, (unsigned long long)lmax);
    }
  }
  __syncthreads();
  {
    int64_t lmax = 0;
    for (int j = tid; j < N; j += kPlanThreads) lmax = max(lmax, colsum[j]);
    lmax = wave_max(lmax);
    if (lane == 0) atomicMax((unsigned long long*)&sh->Lmax, (unsigned long long)lmax);
  }
  __syncthreads();
  if (tid == 0 && sh->err == 0) {
    int64_t den = L.bw_max * P.k_target;
    int64_t tau = (sh->Lmax + den - 1) / den;
    if (tau < 1) tau = 1;
    sh->tau = tau;
    for (int c = 0; c < 3; ++c) {
      int64_t cap = tau * L.bw_cls[c] / P.unit * P.unit;
      if (cap < P.unit) cap = P.unit;
      sh->cap[c] = cap;
      if (cap >= (int64_t(1) << 31)) set_err(sh, VP_ERR_UNSUPPORTED);
    }
    if (sh->total_rem >= (int64_t(1) << 42)) set_err(sh, VP_ERR_UNSUPPORTED);
  }
  __syncthreads();

  // ---------------------------------------------------------------- loop
  while (true) {
    if (sh->err || sh->total_rem == 0) break;
    if (sh->K >= P.k_max) {
      __syncthreads();
      if (tid == 0) set_err(sh, VP_ERR_CAPACITY);
      break;
    }
    const int K = sh->K;

    // Step 1: pattern bases from A, then every shape's score; argmax.
    for (int p = tid; p < NP; p += kPlanThreads) {
      int64_t s = 0;
      const int n = nterms[p];
      for (int m = 0; m < n; ++m) {
        int t = terms[p * L.TS + m];
        if (!(t >> 12)) s += (int64_t)(t & 15) * agg[((t >> 8) & 15) * Q + ((t >> 4) & 15)];
      }
      base[p] = s;
    }
    if (tid == 0) sh->key = 0;
    __syncthreads();
    {
      uint64_t best = 0;
      for (int j = tid; j < L.J0; j += kPlanThreads) {
        uint64_t key = ((uint64_t)base[j] << 20) | (uint64_t)(0xFFFFF - j);
        best = key > best ? key : best;
      }
      if (L.J1 > 0) {
        const int Jr = L.J1 * (nn - 1);
        int k = 1 + tid / L.J1, pp = tid % L.J1;
        const int step_k = kPlanThreads / L.J1, step_p = kPlanThreads % L.J1;
        for (int r = tid; r < Jr; r += kPlanThreads) {
          const int p = L.J0 + pp;
          int64_t s = base[p];
          const int n = nterms[p];
          const int64_t* Bk = agg + k * Q * Q;
          for (int m = 0; m < n; ++m) {
            int t = terms[p * L.TS + m];
            if (t >> 12) s += (int64_t)(t & 15) * Bk[((t >> 8) & 15) * Q + ((t >> 4) & 15)];
          }
          uint64_t key = ((uint64_t)s << 20) | (uint64_t)(0xFFFFF - (L.J0 + r));
          best = key > best ? key : best;
          k += step_k;
          pp += step_p;
          if (pp >= L.J1) {
            pp -= L.J1;
            ++k;
          }
        }
      }
      best = wave_max_u(best);
      if (lane == 0) atomicMax((unsigned long long*)&sh->key, (unsigned long long)best);
    }
    __syncthreads();
    if ((sh->key >> 20) == 0) {
      __syncthreads();
      if (tid == 0) set_err(sh, VP_ERR_NO_PROGRESS);
      break;
    }
    const int jstar = 0xFFFFF - (int)(sh->key & 0xFFFFF);
    int kstar, pstar;
    if (jstar < L.J0) {
      kstar = 0;
      pstar = jstar;
    } else {
      kstar = 1 + (jstar - L.J0) / L.J1;
      pstar = L.J0 + (jstar - L.J0) % L.J1;
    }
    const int lb = cat[L.off_fb + pstar], le = cat[L.off_fe + pstar];
    const int fbase = kstar == 0 ? 0 : L.F0 + (kstar - 1) * L.F1 - L.F0;
    const int fb = lb + fbase, fe = le + fbase;
    if (tid == 0) sh->best_valid = 0;

    // Steps 2-3 over the shape's bucket, FC families at a time.
    for (int cb = fb; cb < fe; cb += P.FC) {
      const int nc = min(P.FC, fe - cb);
      for (int x = tid; x < nc * QG; x += kPlanThreads) {
        const int c = x / QG, idx = x - c * QG, f = cb + c;
        const int lf = kstar == 0 ? f : L.F0 + (f - L.F0) % L.F1;
        cf[c].info[idx] = cat[L.off_fam_info + lf * QG + idx];
        cf[c].outl[idx] = (uint8_t)cat[L.off_fam_out + lf * QG + idx];
        cf[c].inl[idx] = (uint8_t)cat[L.off_fam_in + lf * QG + idx];
        if (idx == 0) {
          cf[c].f = f;
          cf[c].k = kstar;
        }
      }
      __syncthreads();
      // credits h' of every (family, instance, source slot, destination slot)
      {
        const int tot = nc * N;
        int c = tid / N, t = tid - (tid / N) * N;
        const int dc = kPlanThreads / N, dt = kPlanThreads % N;
        for (int x = tid; x < tot; x += kPlanThreads) {
          const int n = rinfo[t] >> 8, idx = t - n * QG;
          const int info = cf[c].info[idx], cl = info & 15;
          const int sg = n * Q + ((info >> 4) & 15);
          const int dn = (cl == VP_PATH_NIC && kstar) ? (n + kstar) % nn : n;
          const int dg = dn * Q + ((info >> 8) & 15);
          const int64_t cap = sh->cap[cl];
          uint32_t* h = hp + ((size_t)c * N + t) * g2;
          for (int il = 0; il < g; ++il)
            for (int jl = 0; jl < g; ++jl) {
              const int i = sg * g + il, j = dg * g + jl;
              uint32_t v = kForbidden;
              if (i != j) {
                int64_t d = P.Drem[(size_t)i * N + j];
                v = (uint32_t)(d < cap ? d : cap);
              }
              h[il * g + jl] = v;
            }
          c += dc;
          t += dt;
          if (t >= N) {
            t -= N;
            ++c;
          }
        }
      }
      __syncthreads();
      for (int pi = wave; pi < nc * NS; pi += kWaves) {
        const int c = pi / NS, s = pi - c * NS;
        Fam fm{&cf[c], rinfo, Q, g, QG, nn, kstar};
        run_pair(P, fm, hp + (size_t)c * N * g2, sl + (size_t)pi * N, dl + (size_t)pi * N, sh, s, K,
                 lane, &pr[pi]);
      }
      __syncthreads();
      // Evaluate (Eq. (9)-(10)) and keep the best family so far.
      if (tid == 0) {
        sh->copy_pair = -1;
        for (int c = 0; c < nc; ++c) {
          int bs = 0;
          for (int s = 1; s < NS; ++s)
            if (pr[c * NS + s].F > pr[c * NS + bs].F) bs = s;
          const PairRes& r = pr[c * NS + bs];
          int64_t xm = 0, bm = 1;
          for (int cl = 0; cl < 3; ++cl)
            if (r.xmax[cl] * bm > xm * L.bw_cls[cl]) {
              xm = r.xmax[cl];
              bm = L.bw_cls[cl];
            }
          if (!sh->best_valid ||
              utility_greater(r.F, xm, bm, sh->best_S, sh->best_xm, sh->best_bm, P.lambda)) {
            sh->best_valid = 1;
            sh->best_S = r.F;
            sh->best_xm = xm;
            sh->best_bm = bm;
            sh->best_f = cb + c;
            sh->best_k = kstar;
            sh->copy_pair = c * NS + bs;
          }
        }
      }
      __syncthreads();
      if (sh->copy_pair >= 0)
        for (int t = tid; t < N; t += kPlanThreads) {
          bsl[t] = sl[(size_t)sh->copy_pair * N + t];
          bdl[t] = dl[(size_t)sh->copy_pair * N + t];
        }
      __syncthreads();
    }

    // Step 4: append E* and subtract X(E*) from D^rem and the aggregates.
    {
      if (tid == 0) sh->S = 0;
      __syncthreads();
      const int f = sh->best_f, k = sh->best_k;
      const int lf = k == 0 ? f : L.F0 + (f - L.F0) % L.F1;
      int64_t served = 0;
      for (int t = tid; t < N; t += kPlanThreads) {
        const int n = rinfo[t] >> 8, idx = t - n * QG;
        const int info = cat[L.off_fam_info + lf * QG + idx], cl = info & 15;
        const int ss = (info >> 4) & 15, ds = (info >> 8) & 15;
        const int dn = (cl == VP_PATH_NIC && k) ? (n + k) % nn : n;
        const int i = (n * Q + ss) * g + bsl[t], j = (dn * Q + ds) * g + bdl[t];
        const int64_t d = P.Drem[(size_t)i * N + j];
        const int64_t x = d < sh->cap[cl] ? d : sh->cap[cl];
        P.Drem[(size_t)i * N + j] = d - x;
        const size_t o = (size_t)K * N + i;
        P.dst[o] = j;
        P.inst[o] = info >> 12;
        P.bytes[o] = x;
        if (x > 0) {
          int kk = dn - n;
          if (kk < 0) kk += nn;
          atomicAdd((unsigned long long*)&agg[(kk * Q + ss) * Q + ds], (unsigned long long)(-x));
        }
        served += x;
      }
      served = wave_sum(served);
      if (lane == 0 && served) atomicAdd((unsigned long long*)&sh->S, (unsigned long long)served);
      __syncthreads();
      if (tid == 0) {
        P.family[K] = f;
        if (sh->S == 0) {
          set_err(sh, VP_ERR_NO_PROGRESS);
        } else {
          sh->total_rem -= sh->S;
          sh->K = K + 1;
        }
      }
      __syncthreads();
    }
  }

  if (tid == 0) {
    *P.K = sh->K;
    if (P.tau) *P.tau = sh->err == VP_ERR_INVALID_DEMAND ? 0 : sh->tau;
    if (sh->err) atomicCAS(P.status, 0, sh->err);
  }
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace

vp_status launch_plan(const PlanLaunch& a, void* stream) {
  const vp_catalog& c = *a.cat;
  const DevCatalogLayout& L = c.lay;
  const int N = L.N, g = L.g, g2 = g * g, NS = a.p.n_start, NP = L.J0 + L.J1;
  if (L.J >= (1 << 20)) return set_error(VP_ERR_UNSUPPORTED, "more than 2^20 shapes");
  if (L.Q * g > kMaxQG) return set_error(VP_ERR_UNSUPPORTED, "too many lanes per node");
  // largest bucket
  int hmax = 1;
  for (int p = 0; p < NP; ++p) hmax = std::max(hmax, c.pat_fe[p] - c.pat_fb[p]);

  PlanArgs P{};
  P.cat = (const int32_t*)c.dev;
  P.L = L;
  P.D = a.demand;
  P.Drem = a.drem;
  P.k_target = a.p.k_target;
  P.lambda = a.p.lambda_ns;
  P.unit = a.p.unit_bytes;
  P.seed = a.p.seed;
  // divisibility by unit = 2^s * odd: low s bits clear and (v >> s) * odd^-1 <= (2^64-1)/odd
  uint64_t u = (uint64_t)a.p.unit_bytes;
  int s = 0;
  while (!(u & 1)) { u >>= 1; ++s; }
  uint64_t inv = u;
  for (int it = 0; it < 6; ++it) inv *= 2 - u * inv;
  P.unit_shift = s;
  P.odd_inv = inv;
  P.odd_lim = ~uint64_t(0) / u;
  P.n_start = NS;
  P.i_aa = a.p.i_aa;
  P.k_max = a.p.k_max;
  P.K = a.K;
  P.family = a.family;
  P.dst = a.dst;
  P.inst = a.inst;
  P.bytes = a.bytes;
  P.tau = a.tau;
  P.status = a.status;

  size_t o = 0;
  P.o_sh = (int32_t)o; o = align_up(o + sizeof(Shared), 16);
  P.o_rinfo = (int32_t)o; o = align_up(o + (size_t)N * 4, 16);
  P.o_agg = (int32_t)o; o = align_up(o + (size_t)L.nn * L.Q * L.Q * 8, 16);
  P.o_terms = (int32_t)o; o = align_up(o + (size_t)NP * L.TS * 2, 16);
  P.o_nterms = (int32_t)o; o = align_up(o + (size_t)NP, 16);
  P.o_base = (int32_t)o; o = align_up(o + (size_t)NP * 8, 16);
  P.o_best = (int32_t)o; o = align_up(o + (size_t)2 * N, 16);
  const size_t fixed = o;
  const size_t per_fam = align_up(sizeof(ChunkFam), 16) + align_up((size_t)NS * sizeof(PairRes), 16) +
                         (size_t)N * g2 * 4 + 2 * align_up((size_t)NS * N, 16);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return set_error(VP_ERR_HIP, "hipGetDevice failed");
  int lds_max = 0;
  if (hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
    return set_error(VP_ERR_HIP, "hipDeviceGetAttribute failed");
  const size_t budget = (size_t)lds_max;
  size_t need_prologue = (size_t)N * 8;   // column sums alias the credit area
  if (fixed + per_fam > budget) return set_error(VP_ERR_UNSUPPORTED, "plan state does not fit in LDS");
  int FC = (int)std::min<size_t>((size_t)hmax, (budget - fixed) / per_fam);
  FC = std::max(FC, 1);
  P.FC = FC;
  P.o_cf = (int32_t)o; o = align_up(o + (size_t)FC * sizeof(ChunkFam), 16);
  P.o_pair = (int32_t)o; o = align_up(o + (size_t)FC * NS * sizeof(PairRes), 16);
  P.o_hp = (int32_t)o; o = align_up(o + std::max((size_t)FC * N * g2 * 4, need_prologue), 16);
  P.o_sl = (int32_t)o; o = align_up(o + (size_t)FC * NS * N, 16);
  P.o_dl = (int32_t)o; o = align_up(o + (size_t)FC * NS * N, 16);
  if (o > budget) return set_error(VP_ERR_UNSUPPORTED, "plan state does not fit in LDS");

  hipStream_t st = (hipStream_t)stream;
  if (hipFuncSetAttribute((const void*)plan_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)o) !=
      hipSuccess)
    return set_error(VP_ERR_HIP, "cannot raise the planner's LDS limit");
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), o, st, P);
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "planner launch failed");
  return VP_OK;
}

}  // namespace vp
