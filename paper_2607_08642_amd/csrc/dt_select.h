// Device building blocks shared by the scan and the expansion kernels:
// order-preserving keys, running log-sum-exp tails, bitonic sorts in LDS and
// the per-row merge of sorted chunk lists (Alg. 1 step 1; section 3.2).
#pragma once

#include "dt_internal.h"

namespace dt {
namespace sel {

// Running tail of exp((x - m) / tau) sums: m is the running max, s the sum.
// c = log2(e) / tau so that exp((x - m) / tau) = exp2((x - m) * c).
struct Tail {
  float m, s;
};

__device__ inline Tail tail_empty() { return Tail{-3.402823466e38f, 0.0f}; }

// 2^x on the hardware unit (v_exp_f32): results below 2^-126 flush to zero,
// which a sum of exponentials relative to its running max can ignore
__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int N>
__device__ inline void tail_add_group(Tail &t, const float (&x)[N], float c) {
  float mx = t.m;
#pragma unroll
  for (int j = 0; j < N; ++j) mx = fmaxf(mx, x[j]);
  float s = t.s * fast_exp2((t.m - mx) * c);
#pragma unroll
  for (int j = 0; j < N; ++j) s += fast_exp2((x[j] - mx) * c);
  t.m = mx;
  t.s = s;
}

__device__ inline void tail_add1(Tail &t, float x, float c) {
  const float xs[1] = {x};
  tail_add_group<1>(t, xs, c);
}

__device__ inline Tail tail_merge(Tail a, Tail b, float c) {
  Tail r;
  r.m = fmaxf(a.m, b.m);
  r.s = a.s * fast_exp2((a.m - r.m) * c) + b.s * fast_exp2((b.m - r.m) * c);
  return r;
}

// Wave-wide reductions with DPP inside each row of 16 lanes (quad swaps, half
// mirror, mirror) and four lane reads across rows; every lane gets the same
// value.  The whole wave must be active.
__device__ inline float readlane_f(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}
template <int CTRL>
__device__ inline float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                               0xF, 0xF, false));
}
template <typename Op>
__device__ inline float wave_reduce(float v, Op op) {
  v = op(v, dpp_f<0xB1>(v));   // quad_perm [1,0,3,2]
  v = op(v, dpp_f<0x4E>(v));   // quad_perm [2,3,0,1]
  v = op(v, dpp_f<0x141>(v));  // row_half_mirror
  v = op(v, dpp_f<0x140>(v));  // row_mirror
  return op(op(readlane_f(v, 0), readlane_f(v, 16)), op(readlane_f(v, 32), readlane_f(v, 48)));
}
// block-wide tail reduction in a fixed order (deterministic); red: NT/64 float2.
// The block max first, then every sum rescaled to it once and added up.
template <int NT>
__device__ inline Tail block_tail(Tail t, float c, float2 *red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  (void)lane;
  const float wm = wave_reduce(t.m, [](float x, float y) { return fmaxf(x, y); });
  if ((threadIdx.x & 63) == 0) red[w].x = wm;
  __syncthreads();
  float m = red[0].x;
#pragma unroll
  for (int i = 1; i < NT / 64; ++i) m = fmaxf(m, red[i].x);
  const float s = wave_reduce(t.s > 0.0f ? t.s * fast_exp2((t.m - m) * c) : 0.0f,
                              [](float x, float y) { return x + y; });
  if ((threadIdx.x & 63) == 0) red[w].y = s;
  __syncthreads();
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) sum += red[i].y;
  __syncthreads();
  return Tail{m, sum};
}

// descending bitonic sort of a wave's 64 values (one per lane)
__device__ inline uint64_t wave_sort_desc(uint64_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const uint64_t p = __shfl_xor(v, j);
      const bool desc = (lane & k) == 0;
      const bool lower = (lane & j) == 0;
      v = (desc == lower) ? (v > p ? v : p) : (v < p ? v : p);
    }
  }
  return v;
}

__host__ __device__ inline int pow2_at_least(int n, int lo) {
  int p = lo;
  while (p < n) p <<= 1;
  return p;
}

// descending bitonic sort of buf[0..P), P a power of two; all NT threads call it
template <int NT>
__device__ void block_sort_desc(uint64_t *buf, int P) {
  const int tid = threadIdx.x;
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int p = tid; p < P / 2; p += NT) {
        const int i = 2 * p - (p & (j - 1));
        const int ixj = i + j;
        const uint64_t a = buf[i], b = buf[ixj];
        const bool desc = (i & k) == 0;
        if (desc ? (a < b) : (a > b)) {
          buf[i] = b;
          buf[ixj] = a;
        }
      }
      __syncthreads();
    }
  }
}

template <bool DEV_SCOPE, typename T>
__device__ inline void put(T *p, T v) {
  if constexpr (DEV_SCOPE)
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    *p = v;
}

// LDS carve of merge_row for nlists lists of M keys (byte offsets)
constexpr int kMergeAllPairs = 1024;  // survivors ranked among themselves up to this many
struct MergeBuf {
  int top, topv, heads, skeys, scnt, sidx, total;
};
__host__ __device__ inline int up16(int b) { return (b + 15) & ~15; }
__host__ __device__ inline MergeBuf merge_buf(int nlists, int M) {
  const int n = nlists * M;
  const int q = (M + nlists - 1) / nlists;
  const int nhp = (nlists * q + 1) & ~1;
  MergeBuf b;
  b.top = up16(8 * n);                 // keys: n u64 at 0
  b.topv = up16(b.top + 8 * M);        // top: M u64
  b.heads = up16(b.topv + 4 * M);      // topv: M f32
  b.skeys = up16(b.heads + 8 * nhp);   // heads: nhp u64
  const int ns_cap = n < kMergeAllPairs ? n : kMergeAllPairs;
  b.scnt = up16(b.skeys + 8 * (ns_cap + 2));  // skeys: survivors' keys (+ padding)
  b.sidx = up16(b.scnt + 4 * n);       // scnt: n i32
  b.total = up16(b.sidx + 2 * n);      // sidx: n i16
  return b;
}
__host__ __device__ inline int merge_buf_bytes(int nlists, int M) { return merge_buf(nlists, M).total; }

// Merge the sorted chunk lists of one row: the row's M best keys and
// R = log sum over every other element of exp(x / tau).
//   lists: nlists * M keys (0 = empty slot), each list sorted descending;
//   tails: per-chunk (max, sum) of the elements not in its list; flags: per chunk.
// Exact without sorting the lists together:
//  * thr = the M-th best of the first q = ceil(M / nlists) keys of every list.
//    Those keys are all in the row, so at least M keys are >= thr and thr is
//    <= the row's M-th best key: keys below thr go straight to the tail.
//  * a surviving key's rank below M is the number of larger survivors: a key
//    outside every list lies below the M keys of its chunk's list, and a list
//    key above a survivor is a survivor itself.  (With very many survivors the
//    rank is its position in its own list plus a binary search in every other
//    list, exact in the same way.)
// Every key joins the tail through the thread that holds its list position,
// so the result does not depend on the order the survivors were collected in.
// buf: merge_buf_bytes(nlists, M) bytes of LDS; red: NT/64 float2.
// DEV_SCOPE selects device-scope stores (results read by other workgroups).
// vadd (nullable): candv[m] = logit + vadd[cand[m]] instead of the logit.
template <int NT, bool DEV_SCOPE>
__device__ __attribute__((always_inline)) void merge_row(const uint64_t *lists, int nlists, int M, const float2 *tails,
                          const int32_t *flags, float c, float inv_tau, uint64_t *buf,
                          float2 *red, int *flag_lds, int32_t *cand, float *candv, float *tailR,
                          int32_t *rflag, const float *vadd) {
  const int tid = threadIdx.x;
  const int n = nlists * M;
  const int q = (M + nlists - 1) / nlists;
  const int nh = nlists * q, nhp = (nh + 1) & ~1;
  const MergeBuf mb = merge_buf(nlists, M);
  char *base = reinterpret_cast<char *>(buf);
  uint64_t *keys = buf;                                           // [n]
  uint64_t *top = reinterpret_cast<uint64_t *>(base + mb.top);    // [M]
  float *topv = reinterpret_cast<float *>(base + mb.topv);        // [M]
  uint64_t *heads = reinterpret_cast<uint64_t *>(base + mb.heads);  // [nhp]
  uint64_t *skeys = reinterpret_cast<uint64_t *>(base + mb.skeys);  // survivors' keys
  int32_t *scnt = reinterpret_cast<int32_t *>(base + mb.scnt);    // [n] survivor ranks
  int16_t *sidx = reinterpret_cast<int16_t *>(base + mb.sidx);    // [n] survivor positions
  __shared__ uint64_t s_thr;
  __shared__ int s_ns;
  if (tid == 0) {
    *flag_lds = 0;
    s_ns = 0;
    s_thr = 1;  // stays 1 (keep every key) when the heads hold fewer than M keys
    if (nh & 1) heads[nh] = 0ull;
  }
  // 0. one round trip: the lists (heads copied on the way), chunk tails and flags
  Tail t = tail_empty();
  int bad = 0;
  {
    float2 tl = make_float2(0.0f, 0.0f);
    if (tid < nlists) {
      tl = tails[tid];
      bad = flags[tid];
    }
    for (int i0 = 0; i0 < n; i0 += 4 * NT) {
      uint64_t v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = i0 + u * NT + tid;
        v[u] = i < n ? lists[i] : 0ull;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = i0 + u * NT + tid;
        if (i < n) {
          keys[i] = v[u];
          const int l = i / M, p = i - l * M;
          if (p < q) heads[l * q + p] = v[u];
        }
      }
    }
    if (tid < nlists) t = tail_merge(t, Tail{tl.x, tl.y}, c);
    for (int i = tid + NT; i < nlists; i += NT) {
      t = tail_merge(t, Tail{tails[i].x, tails[i].y}, c);
      bad |= flags[i];
    }
  }
  for (int i = tid; i < M; i += NT) top[i] = 0ull;
  for (int i = tid; i < nh; i += NT) scnt[i] = 0;
  __syncthreads();
  if (bad) atomicOr(flag_lds, bad);
  // 1. thr: the M-th largest head (q heads per list); each head's count of
  //    larger heads is split over RS threads
  {
    const int np = nhp / 2;
    const int RS = nh >= NT ? 1 : (NT / nh > 16 ? 16 : NT / nh);
    const int per = (np + RS - 1) / RS;
    const ulonglong2 *h2 = reinterpret_cast<const ulonglong2 *>(heads);
    for (int p = tid; p < nh * RS; p += NT) {
      const int h = p / RS, j0 = (p - h * RS) * per;
      const int j1 = j0 + per < np ? j0 + per : np;
      const uint64_t k = heads[h];
      int r = 0;
#pragma unroll 4
      for (int j = j0; j < j1; ++j) {
        const ulonglong2 v = h2[j];
        r += (v.x > k) + (v.y > k);
      }
      if (r) atomicAdd(&scnt[h], r);
    }
    __syncthreads();
    for (int h = tid; h < nh; h += NT)
      if (heads[h] && scnt[h] == M - 1) s_thr = heads[h];
  }
  __syncthreads();
  const uint64_t thr = s_thr;
  // 2. survivors (keys >= thr) start from their own position; the rest feed the tail
  for (int i = tid; i < n; i += NT) {
    const uint64_t k = keys[i];
    if (!k) continue;
    if (k >= thr) {
      const int at = atomicAdd(&s_ns, 1);
      sidx[at] = (int16_t)i;
      scnt[at] = i % M;
      if (at < kMergeAllPairs) skeys[at] = k;
    } else {
      tail_add1(t, key_value(k), c);
    }
  }
  __syncthreads();
  const int ns = s_ns;
  // 3. rank the survivors; the M best go to top[] and leave keys[] (zeroed)
  if (ns <= kMergeAllPairs) {
    // every key above a survivor is itself a survivor or lies below M keys of
    // its own list, so a survivor's rank among the survivors is its rank in
    // the row whenever that is below M.  Each count is split over RS threads.
    if (tid == 0 && (ns & 1)) skeys[ns] = 0ull;  // pad for paired reads
    for (int sv = tid; sv < ns; sv += NT) scnt[sv] = 0;
    // the first survivor this thread places: its vadd entry is in flight during the count
    const float va0 = (vadd && tid < ns) ? vadd[key_index(skeys[tid])] : 0.0f;
    __syncthreads();
    const int np = (ns + 1) >> 1;
    const int RS = ns >= NT ? 1 : (NT / ns > 16 ? 16 : NT / ns);
    const int per = (np + RS - 1) / RS;
    const ulonglong2 *s2 = reinterpret_cast<const ulonglong2 *>(skeys);
    for (int p = tid; p < ns * RS; p += NT) {
      const int sv = p / RS, j0 = (p - sv * RS) * per;
      const int j1 = j0 + per < np ? j0 + per : np;
      const uint64_t k = skeys[sv];
      int r = 0;
#pragma unroll 4
      for (int j = j0; j < j1; ++j) {
        const ulonglong2 kk = s2[j];
        r += (kk.x > k) + (kk.y > k);
      }
      if (r) atomicAdd(&scnt[sv], r);
    }
    __syncthreads();
    for (int sv = tid; sv < ns; sv += NT) {
      const int r = scnt[sv];
      if (r < M) {
        const uint64_t k = skeys[sv];
        const float va = sv == tid ? va0 : (vadd ? vadd[key_index(k)] : 0.0f);
        top[r] = k;
        topv[r] = key_value(k) + va;
        keys[sidx[sv]] = 0ull;
      }
    }
  } else {
    // + the larger keys of every other list: one binary search per (survivor, list)
    for (int p = tid; p < ns * nlists; p += NT) {
      const int sv = p / nlists, j = p % nlists;
      const int i = sidx[sv];
      if (j == i / M) continue;
      const uint64_t k = keys[i];
      const uint64_t *lj = keys + j * M;
      int lo = 0, hi = M;  // count of lj[] > k (lj is descending)
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (lj[mid] > k)
          lo = mid + 1;
        else
          hi = mid;
      }
      if (lo) atomicAdd(&scnt[sv], lo);
    }
    __syncthreads();
    for (int sv = tid; sv < ns; sv += NT) {
      const int r = scnt[sv];
      if (r < M) {
        const uint64_t k = keys[sidx[sv]];
        top[r] = k;
        topv[r] = key_value(k) + (vadd ? vadd[key_index(k)] : 0.0f);
      }
    }
    __syncthreads();
    for (int sv = tid; sv < ns; sv += NT)
      if (scnt[sv] < M) keys[sidx[sv]] = 0ull;
  }
  __syncthreads();
  // 4. survivors outside the M best join the tail from their list position
  for (int i = tid; i < n; i += NT) {
    const uint64_t k = keys[i];
    if (k >= thr) tail_add1(t, key_value(k), c);  // thr >= 1: empty slots stay out
  }
  t = block_tail<NT>(t, c, red);
  for (int i = tid; i < M; i += NT) {
    const uint64_t k = top[i];
    put<DEV_SCOPE>(cand + i, k ? (int32_t)key_index(k) : (int32_t)-1);
    put<DEV_SCOPE>(candv + i, k ? topv[i] : -__builtin_huge_valf());
  }
  if (tid == 0) {
    put<DEV_SCOPE>(tailR, t.s > 0.0f ? t.m * inv_tau + logf(t.s) : -__builtin_huge_valf());
    put<DEV_SCOPE>(rflag, (int32_t)(*flag_lds ? DT_TREE_NONFINITE : 0));
  }
  __syncthreads();
}

}  // namespace sel
}  // namespace dt
