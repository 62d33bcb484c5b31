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

// SHIFT: the row's candidate values and R are written less the row's largest
// value s0 (R less s0 / tau), which changes no log-probability (a constant
// per row) but keeps the consumer's sums of a value and a correction at the
// magnitude of their difference: logits offset by thousands would otherwise
// leave fp32 ulps of 1e-4 in every score.  (s0 = 0 for a row whose largest
// value is not finite.)
__device__ inline float row_shift(float top) { return __builtin_isfinite(top) ? top : 0.0f; }

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
template <int NT, bool DEV_SCOPE, bool SHIFT = false>
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
  const float s0 = SHIFT && top[0] ? row_shift(key_value(top[0])) : 0.0f;
  for (int i = tid; i < M; i += NT) {
    const uint64_t k = top[i];
    put<DEV_SCOPE>(cand + i, k ? (int32_t)key_index(k) : (int32_t)-1);
    float v = k ? topv[i] : -__builtin_huge_valf();
    if (SHIFT && k) v = (key_value(k) - s0) + (vadd ? vadd[key_index(k)] : 0.0f);
    put<DEV_SCOPE>(candv + i, v);
  }
  if (tid == 0) {
    put<DEV_SCOPE>(tailR, t.s > 0.0f ? (t.m - s0) * inv_tau + logf(t.s) : -__builtin_huge_valf());
    put<DEV_SCOPE>(rflag, (int32_t)(*flag_lds ? DT_TREE_NONFINITE : 0));
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// One wave merges a row's segment lists when M <= 64 and there are at most 16
// lists: lane p holds position p of every list, and pairs of lists combine in
// a tree.  Of a descending list A and an ascending list B, max(A[i], B[i]) is
// the better half of A and B as a bitonic sequence (six compare-exchange
// stages sort it) and min(A[i], B[i]) the worse half, which joins the lane's
// tail right away: every key not among the row's M best is added to exactly
// one lane's tail, in an order fixed by the tree.  No LDS and no barrier.

// a 64-bit value from lane ^ J (DPP inside rows of 16 lanes, swizzle across
// rows, permute across halves); the whole wave must be active
template <int J>
__device__ inline uint64_t lane_xor64(uint64_t v) {
  const int lo = (int)(uint32_t)v, hi = (int)(uint32_t)(v >> 32);
  int plo, phi;
  if constexpr (J == 1 || J == 2 || J == 8) {
    // quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_ror:8
    constexpr int ctrl = J == 1 ? 0xB1 : (J == 2 ? 0x4E : 0x128);
    plo = __builtin_amdgcn_update_dpp(0, lo, ctrl, 0xF, 0xF, false);
    phi = __builtin_amdgcn_update_dpp(0, hi, ctrl, 0xF, 0xF, false);
  } else if constexpr (J == 4) {
    // row_shl:4 (from lane + 4) where bit 2 is clear, row_shr:4 (lane - 4) where set
    const bool up = (threadIdx.x & 4) != 0;
    const int lo_a = __builtin_amdgcn_update_dpp(0, lo, 0x104, 0xF, 0xF, false);
    const int lo_b = __builtin_amdgcn_update_dpp(0, lo, 0x114, 0xF, 0xF, false);
    const int hi_a = __builtin_amdgcn_update_dpp(0, hi, 0x104, 0xF, 0xF, false);
    const int hi_b = __builtin_amdgcn_update_dpp(0, hi, 0x114, 0xF, 0xF, false);
    plo = up ? lo_b : lo_a;
    phi = up ? hi_b : hi_a;
  } else if constexpr (J == 16) {
    // swizzle bit mode inside 32 lanes: and 0x1F, or 0, xor 0x10
    plo = __builtin_amdgcn_ds_swizzle(lo, 0x401F);
    phi = __builtin_amdgcn_ds_swizzle(hi, 0x401F);
  } else {
    static_assert(J == 32, "lane distance");
    const int a = (int)((threadIdx.x & 63) ^ 32) * 4;
    plo = __builtin_amdgcn_ds_bpermute(a, lo);
    phi = __builtin_amdgcn_ds_bpermute(a, hi);
  }
  return ((uint64_t)(uint32_t)phi << 32) | (uint32_t)plo;
}

template <int J>
__device__ inline uint64_t cx_stage(uint64_t v, bool desc) {
  const uint64_t p = lane_xor64<J>(v);
  const bool keep_max = ((threadIdx.x & J) == 0) == desc;
  return ((p > v) == keep_max) ? p : v;  // (equal keys are both empty)
}

// sorts a bitonic sequence of 64 keys (one per lane), descending or ascending
__device__ inline uint64_t bitonic_clean64(uint64_t v, bool desc) {
  v = cx_stage<32>(v, desc);
  v = cx_stage<16>(v, desc);
  v = cx_stage<8>(v, desc);
  v = cx_stage<4>(v, desc);
  v = cx_stage<2>(v, desc);
  return cx_stage<1>(v, desc);
}

// the better half of a descending list a and an ascending list b, sorted in
// direction desc; the worse half joins the lane's tail (empty slots add
// nothing: -inf, whose term is 0 against any reference the tail can hold --
// the least being -FLT_MAX, against which -FLT_MAX itself would add 1)
__device__ inline uint64_t merge_halves(uint64_t a, uint64_t b, bool desc, Tail &t, float c) {
  const bool ga = a > b;
  const uint64_t hi = ga ? a : b, lo = ga ? b : a;
  tail_add1(t, lo ? key_value(lo) : -__builtin_huge_valf(), c);
  return bitonic_clean64(hi, desc);
}

// full bitonic sort of 64 keys (one per lane), descending or ascending
__device__ inline uint64_t wave_sort64(uint64_t v, bool desc) {
  const int lane = threadIdx.x & 63;
  // a stage of block size k orders each k-block the way the next block size needs
  auto dir = [&](int k) { return ((lane & k) == 0) == desc; };
  v = cx_stage<1>(v, dir(2));
  v = cx_stage<2>(v, dir(4));
  v = cx_stage<1>(v, dir(4));
  v = cx_stage<4>(v, dir(8));
  v = cx_stage<2>(v, dir(8));
  v = cx_stage<1>(v, dir(8));
  v = cx_stage<8>(v, dir(16));
  v = cx_stage<4>(v, dir(16));
  v = cx_stage<2>(v, dir(16));
  v = cx_stage<1>(v, dir(16));
  v = cx_stage<16>(v, dir(32));
  v = cx_stage<8>(v, dir(32));
  v = cx_stage<4>(v, dir(32));
  v = cx_stage<2>(v, dir(32));
  v = cx_stage<1>(v, dir(32));
  return bitonic_clean64(v, desc);
}

constexpr int kWaveMergeLists = 16;

__host__ __device__ inline bool wave_merge_fits(int nlists, int M) {
  return M <= 64 && nlists <= kWaveMergeLists;
}

// The same results as merge_row (the row's M best keys, R over the rest, the
// row flag), computed by the calling wave alone; wave_merge_fits must hold.
template <bool DEV_SCOPE, bool SHIFT = false>
__device__ __attribute__((always_inline)) void merge_row_wave(
    const uint64_t *lists, int nlists, int M, const float2 *tails, const int32_t *flags, float c,
    float inv_tau, int32_t *cand, float *candv, float *tailR, int32_t *rflag, const float *vadd) {
  constexpr int NL = kWaveMergeLists;
  const int lane = threadIdx.x & 63;
  // lists at even positions of the tree descending, odd ones reversed (ascending)
  uint64_t k[NL];
#pragma unroll
  for (int j = 0; j < NL; ++j) {
    const int pos = (j & 1) ? 63 - lane : lane;
    k[j] = (j < nlists && pos < M) ? lists[j * M + pos] : 0ull;
  }
  Tail t = tail_empty();
  int bad = 0;
  if (lane < nlists) {
    const float2 tl = tails[lane];
    t = Tail{tl.x, tl.y};
    bad = flags[lane];
  }
  // level s: k[j] (j a multiple of 2s) takes the best 64 of lists j .. j+2s-1,
  // descending when it is the left operand of the next level, else ascending
#pragma unroll
  for (int s = 1; s < NL; s <<= 1) {
#pragma unroll
    for (int j = 0; j < NL; j += 2 * s) {
      if (j >= nlists) break;
      const bool desc = ((j / (2 * s)) & 1) == 0;
      if (j + s < nlists) {
        k[j] = merge_halves(k[j], k[j + s], desc, t, c);
      } else if (!desc) {
        k[j] = bitonic_clean64(k[j], false);  // a lone list, now the right operand
      }
    }
  }
  const uint64_t top = k[0];
  const bool keep = lane < M && top != 0ull;
  if (lane >= M && top) tail_add1(t, key_value(top), c);
  const float va = (keep && vadd) ? vadd[key_index(top)] : 0.0f;
  // the tail: the wave's max, then every lane's sum rescaled to it once
  const float m = wave_reduce(t.m, [](float x, float y) { return fmaxf(x, y); });
  const float sum = wave_reduce(t.s > 0.0f ? t.s * fast_exp2((t.m - m) * c) : 0.0f,
                                [](float x, float y) { return x + y; });
  const bool any_bad = __ballot(bad != 0) != 0ull;
  const float s0 = SHIFT ? row_shift(readlane_f(top ? key_value(top) : 0.0f, 0)) : 0.0f;
  if (lane < M) {
    put<DEV_SCOPE>(cand + lane, keep ? (int32_t)key_index(top) : (int32_t)-1);
    put<DEV_SCOPE>(candv + lane, keep ? (key_value(top) - s0) + va : -__builtin_huge_valf());
  }
  if (lane == 0) {
    put<DEV_SCOPE>(tailR, sum > 0.0f ? (m - s0) * inv_tau + logf(sum) : -__builtin_huge_valf());
    put<DEV_SCOPE>(rflag, (int32_t)(any_bad ? DT_TREE_NONFINITE : 0));
  }
}

// The same merge spread over the NT / 64 waves of a workgroup (every thread
// calls it): wave w merges lists 2w and 2w + 1, then the tree's levels meet in
// LDS (xbuf: NT keys), one barrier each; the tails combine as in block_tail.
template <bool DEV_SCOPE, int NT, bool SHIFT = false>
__device__ __attribute__((always_inline)) void merge_row_tree(
    const uint64_t *lists, int nlists, int M, const float2 *tails, const int32_t *flags, float c,
    float inv_tau, uint64_t *xbuf, float2 *red, int32_t *cand, float *candv, float *tailR,
    int32_t *rflag, const float *vadd) {
  constexpr int W = NT / 64;
  static_assert(2 * W >= kWaveMergeLists, "two lists per wave");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = 2 * wave;  // this wave's first list; the tree as in merge_row_wave
  Tail t = tail_empty();
  int bad = 0;
  if (wave == 0 && lane < nlists) {
    const float2 tl = tails[lane];
    t = Tail{tl.x, tl.y};
    bad = flags[lane];
  }
  uint64_t v = 0ull;
  if (j < nlists) {
    const uint64_t a = lane < M ? lists[j * M + lane] : 0ull;
    const bool desc = (wave & 1) == 0;
    if (j + 1 < nlists) {
      const uint64_t b = 63 - lane < M ? lists[(j + 1) * M + 63 - lane] : 0ull;
      v = merge_halves(a, b, desc, t, c);
    } else {
      v = desc ? a : bitonic_clean64(a, false);
    }
  }
#pragma unroll
  for (int s = 2; s < 2 * W; s <<= 1) {
    // right operands publish; a slot read at this level is never written at the next
    if (j < nlists && (j % (2 * s)) == s) xbuf[wave * 64 + lane] = v;
    __syncthreads();
    if (j < nlists && (j % (2 * s)) == 0) {
      const bool desc = ((j / (2 * s)) & 1) == 0;
      if (j + s < nlists)
        v = merge_halves(v, xbuf[(wave + s / 2) * 64 + lane], desc, t, c);
      else if (!desc)
        v = bitonic_clean64(v, false);
    }
  }
  const bool keep = wave == 0 && lane < M && v != 0ull;
  if (wave == 0 && lane >= M && v) tail_add1(t, key_value(v), c);
  const float va = (keep && vadd) ? vadd[key_index(v)] : 0.0f;
  const bool any_bad = __ballot(bad != 0) != 0ull;  // (wave 0 holds the flags)
  t = block_tail<NT>(t, c, red);
  if (wave == 0) {
    const float s0 = SHIFT ? row_shift(readlane_f(v ? key_value(v) : 0.0f, 0)) : 0.0f;
    if (lane < M) {
      put<DEV_SCOPE>(cand + lane, keep ? (int32_t)key_index(v) : (int32_t)-1);
      put<DEV_SCOPE>(candv + lane, keep ? (key_value(v) - s0) + va : -__builtin_huge_valf());
    }
    if (lane == 0) {
      put<DEV_SCOPE>(tailR, t.s > 0.0f ? (t.m - s0) * inv_tau + logf(t.s) : -__builtin_huge_valf());
      put<DEV_SCOPE>(rflag, (int32_t)(any_bad ? DT_TREE_NONFINITE : 0));
    }
  }
}

}  // namespace sel
}  // namespace dt
