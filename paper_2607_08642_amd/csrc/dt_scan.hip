// S1: per-depth marginal top-M and the tail log-sum-exp (Alg. 1 step 1;
// section 3.2, candidate restriction).
//
// Every logit row [V] is split into chunks; one 256-thread workgroup streams a
// chunk through an exact top-M selector and writes the chunk's M best keys plus
// the (max, sum-exp) of every other element of the chunk.  A second kernel runs
// the same selector over the chunk candidates of a row and folds the chunk
// tails, giving the row's top-M and R = log sum_{v not in top-M} exp(x_v/tau).
//
// Keys are 64-bit (order-preserving value bits, ~index), so the total order
// (value desc, id asc) is a plain integer order with no ties.  The selector
// keeps a sorted list of the best M keys in LDS and a buffer of new candidates
// that beat the current threshold; when the buffer grows past a bound the
// union is bitonic-sorted and cut back to M.  The first threshold is an exact
// lower bound on the chunk's M-th best key: every wave sorts its 64 per-lane
// maxima and takes the ceil(M/4)-th, and the minimum over the 4 waves leaves at
// least M elements at or above it.  Elements below the threshold go straight
// into the running tail sum; keys evicted by a flush join it then.
#include "dt_internal.h"

namespace dt {

namespace {

constexpr int kWaves = kScanThreads / 64;

struct SelLDS {
  uint64_t buf[kScanSortCap];
  uint64_t wthr[kWaves];
  float2 red[kWaves];
  int nbuf;
  int nlist;
  int flag;
  uint64_t thr;
};

struct Tail {
  float m, s;
};

__device__ inline void tail_init(Tail &t) {
  t.m = -3.402823466e38f;
  t.s = 0.0f;
}

// fold a group of values (already masked to -inf where not counted)
template <int N>
__device__ inline void tail_add_group(Tail &t, const float (&x)[N], float c) {
  float mx = t.m;
#pragma unroll
  for (int j = 0; j < N; ++j) mx = fmaxf(mx, x[j]);
  float s = t.s * exp2f((t.m - mx) * c);
#pragma unroll
  for (int j = 0; j < N; ++j) s += exp2f((x[j] - mx) * c);
  t.m = mx;
  t.s = s;
}

__device__ inline void tail_add1(Tail &t, float x, float c) {
  float xs[1] = {x};
  tail_add_group<1>(t, xs, c);
}

__device__ inline Tail tail_merge(Tail a, Tail b, float c) {
  Tail r;
  r.m = fmaxf(a.m, b.m);
  r.s = a.s * exp2f((a.m - r.m) * c) + b.s * exp2f((b.m - r.m) * c);
  return r;
}

__device__ inline Tail block_tail(SelLDS &sh, Tail t, float c) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    Tail u;
    u.m = __shfl_xor(t.m, o);
    u.s = __shfl_xor(t.s, o);
    t = tail_merge(t, u, c);
  }
  if (lane == 0) sh.red[w] = make_float2(t.m, t.s);
  __syncthreads();
  Tail r;
  r.m = sh.red[0].x;
  r.s = sh.red[0].y;
  for (int i = 1; i < kWaves; ++i) {
    Tail u;
    u.m = sh.red[i].x;
    u.s = sh.red[i].y;
    r = tail_merge(r, u, c);
  }
  __syncthreads();
  return r;
}

// descending bitonic sort of a wave's 64 values (one per lane)
__device__ inline uint64_t wave_sort_desc(uint64_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      uint64_t p = __shfl_xor(v, j);
      bool desc = (lane & k) == 0;
      bool lower = (lane & j) == 0;
      v = (desc == lower) ? (v > p ? v : p) : (v < p ? v : p);
    }
  }
  return v;
}

__device__ inline int next_pow2(int n) {
  int p = 64;
  while (p < n) p <<= 1;
  return p;
}

// sort buf[0..nbuf) descending, keep the best M as the list, evict the rest
__device__ void flush(SelLDS &sh, int M, Tail &tail, float c) {
  const int tid = threadIdx.x;
  const int n = sh.nbuf;
  const int P = next_pow2(n);
  for (int i = n + tid; i < P; i += kScanThreads) sh.buf[i] = 0;
  __syncthreads();
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int p = tid; p < P / 2; p += kScanThreads) {
        int i = 2 * p - (p & (j - 1));
        int ixj = i + j;
        uint64_t a = sh.buf[i], b = sh.buf[ixj];
        bool desc = (i & k) == 0;
        if (desc ? (a < b) : (a > b)) {
          sh.buf[i] = b;
          sh.buf[ixj] = a;
        }
      }
      __syncthreads();
    }
  }
  for (int i = M + tid; i < n; i += kScanThreads) tail_add1(tail, key_value(sh.buf[i]), c);
  __syncthreads();
  if (tid == 0) {
    int nl = n < M ? n : M;
    sh.nlist = nl;
    sh.nbuf = nl;
    if (nl == M) {
      uint64_t t = sh.buf[M - 1] + 1;
      if (t > sh.thr) sh.thr = t;
    }
  }
  __syncthreads();
}

// One sub-batch: EPT keys per thread (0 = no element).  `first` computes the
// initial threshold from the per-lane maxima.
template <int EPT>
__device__ void select_batch(SelLDS &sh, const uint64_t (&key)[EPT], const float (&val)[EPT],
                             bool first, int M, Tail &tail, float c) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (first) {
    uint64_t mx = 0;
#pragma unroll
    for (int j = 0; j < EPT; ++j) mx = key[j] > mx ? key[j] : mx;
    uint64_t srt = wave_sort_desc(mx);
    int q = (M + kWaves - 1) / kWaves;  // <= 64 since M <= 256
    uint64_t tq = __shfl(srt, q - 1);
    if (lane == 0) sh.wthr[w] = tq;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint64_t t = sh.wthr[0];
      for (int i = 1; i < kWaves; ++i) t = sh.wthr[i] < t ? sh.wthr[i] : t;
      if (t == 0) t = 1;  // fewer than M elements so far: accept everything
      if (t > sh.thr) sh.thr = t;
    }
    __syncthreads();
  }
  const uint64_t thr = sh.thr;
  float tv[EPT];
  uint64_t bal[EPT];
  int tot = 0;
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    bool pass = key[j] != 0 && key[j] >= thr;
    tv[j] = (key[j] != 0 && !pass) ? val[j] : -__builtin_huge_valf();
    bal[j] = __ballot(pass);
    tot += __popcll(bal[j]);
  }
  tail_add_group<EPT>(tail, tv, c);
  if (tot) {
    int base = 0;
    if (lane == 0) base = atomicAdd(&sh.nbuf, tot);
    base = __shfl(base, 0);
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      if ((bal[j] >> lane) & 1ull) sh.buf[base + __popcll(bal[j] & below)] = key[j];
      base += __popcll(bal[j]);
    }
  }
  __syncthreads();
  if (sh.nbuf - sh.nlist > kScanFlushAt) flush(sh, M, tail, c);
}

__device__ inline void init_sel(SelLDS &sh) {
  if (threadIdx.x == 0) {
    sh.nbuf = 0;
    sh.nlist = 0;
    sh.flag = 0;
    sh.thr = 1;
  }
  __syncthreads();
}

__device__ inline bool nonfinite(float v) { return v != v || v == __builtin_huge_valf(); }

template <typename T>
struct Elem;
template <>
struct Elem<uint16_t> {
  static constexpr int EPT = 8;
};
template <>
struct Elem<float> {
  static constexpr int EPT = 4;
};

template <typename T>
__device__ inline float to_f32(T x);
template <>
__device__ inline float to_f32<uint16_t>(uint16_t x) {
  return bf16_to_f32(x);
}
template <>
__device__ inline float to_f32<float>(float x) {
  return x;
}

// K1: top-M of one chunk of one row
template <typename T, bool VEC>
__global__ __launch_bounds__(kScanThreads) void scan_chunk_kernel(const T *__restrict__ logits,
                                                                  ScanGeom g, float c,
                                                                  uint64_t *__restrict__ ckeys,
                                                                  float2 *__restrict__ ctail,
                                                                  int32_t *__restrict__ cflag) {
  constexpr int EPT = Elem<T>::EPT;
  constexpr int UNR = 4;  // sub-batches whose loads are issued together
  __shared__ SelLDS sh;
  const int tid = threadIdx.x;
  const int row = blockIdx.y, chunk = blockIdx.x;
  const int start = chunk * g.chunk;
  const int n = min(g.chunk, g.V - start);
  const T *base = logits + (size_t)row * g.V + start;
  init_sel(sh);
  Tail tail;
  tail_init(tail);
  int bad = 0;
  const int step = kScanThreads * EPT;
  bool first = true;
  for (int b0 = 0; b0 < n; b0 += step * UNR) {
    float v[UNR][EPT];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int off = b0 + u * step + tid * EPT;
      if (VEC && off + EPT <= n) {
        if constexpr (EPT == 8) {
          uint4 r = *reinterpret_cast<const uint4 *>(base + off);
          uint32_t w4[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            v[u][2 * q] = __uint_as_float(w4[q] << 16);
            v[u][2 * q + 1] = __uint_as_float(w4[q] & 0xFFFF0000u);
          }
        } else {
          float4 r = *reinterpret_cast<const float4 *>(base + off);
          v[u][0] = r.x;
          v[u][1] = r.y;
          v[u][2] = r.z;
          v[u][3] = r.w;
        }
      } else {
#pragma unroll
        for (int j = 0; j < EPT; ++j)
          v[u][j] = (off + j < n) ? to_f32<T>(base[off + j]) : __builtin_nanf("");
      }
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      if (b0 + u * step >= n) break;  // uniform
      const int off = b0 + u * step + tid * EPT;
      uint64_t key[EPT];
      float val[EPT];
#pragma unroll
      for (int j = 0; j < EPT; ++j) {
        const bool in = off + j < n;
        float x = v[u][j];
        if (in && nonfinite(x)) bad = 1;
        // NaN / +inf make the row invalid; keep them out of the arithmetic
        if (!in || nonfinite(x)) {
          key[j] = 0;
          val[j] = 0.0f;
        } else {
          key[j] = make_key(x, (uint32_t)(start + off + j));
          val[j] = x;
        }
      }
      select_batch<EPT>(sh, key, val, first, g.M, tail, c);
      first = false;
    }
  }
  if (sh.nbuf > sh.nlist) flush(sh, g.M, tail, c);
  if (bad) atomicOr(&sh.flag, 1);
  Tail t = block_tail(sh, tail, c);
  const size_t cidx = (size_t)row * g.nchunks + chunk;
  uint64_t *out = ckeys + cidx * g.M;
  for (int i = tid; i < g.M; i += kScanThreads) out[i] = i < sh.nlist ? sh.buf[i] : 0ull;
  if (tid == 0) {
    ctail[cidx] = make_float2(t.m, t.s);
    cflag[cidx] = sh.flag ? DT_TREE_NONFINITE : 0;
  }
}

// K2: merge the chunk candidates of one row
__global__ __launch_bounds__(kScanThreads) void scan_merge_kernel(
    ScanGeom g, float c, float inv_tau, const uint64_t *__restrict__ ckeys,
    const float2 *__restrict__ ctail, const int32_t *__restrict__ cflag, int32_t *__restrict__ cand,
    float *__restrict__ candv, float *__restrict__ tailR, int32_t *__restrict__ rflag) {
  constexpr int EPT = 8;
  __shared__ SelLDS sh;
  const int tid = threadIdx.x;
  const int row = blockIdx.x;
  init_sel(sh);
  Tail tail;
  tail_init(tail);
  int bad = 0;
  for (int i = tid; i < g.nchunks; i += kScanThreads) {
    const float2 ct = ctail[(size_t)row * g.nchunks + i];
    Tail u;
    u.m = ct.x;
    u.s = ct.y;
    tail = tail_merge(tail, u, c);
    bad |= cflag[(size_t)row * g.nchunks + i];
  }
  const uint64_t *in = ckeys + (size_t)row * g.nchunks * g.M;
  const int n = g.nchunks * g.M;
  const int step = kScanThreads * EPT;
  bool first = true;
  for (int b0 = 0; b0 < n; b0 += step) {
    uint64_t key[EPT];
    float val[EPT];
    const int off = b0 + tid * EPT;
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      key[j] = (off + j < n) ? in[off + j] : 0ull;
      val[j] = key[j] ? key_value(key[j]) : 0.0f;
    }
    select_batch<EPT>(sh, key, val, first, g.M, tail, c);
    first = false;
  }
  if (sh.nbuf > sh.nlist) flush(sh, g.M, tail, c);
  if (bad) atomicOr(&sh.flag, 1);
  Tail t = block_tail(sh, tail, c);
  for (int i = tid; i < g.M; i += kScanThreads) {
    const uint64_t k = i < sh.nlist ? sh.buf[i] : 0ull;
    cand[(size_t)row * g.M + i] = k ? (int32_t)key_index(k) : -1;
    candv[(size_t)row * g.M + i] = k ? key_value(k) : -__builtin_huge_valf();
  }
  if (tid == 0) {
    tailR[row] = t.s > 0.0f ? t.m * inv_tau + logf(t.s) : -__builtin_huge_valf();
    rflag[row] = sh.flag ? DT_TREE_NONFINITE : 0;
  }
}

}  // namespace

ScanGeom scan_geom(int rows, int V, int M) {
  ScanGeom g;
  g.rows = rows;
  g.V = V;
  g.M = M;
  // aim for ~4 workgroups per CU over the whole call; chunks are multiples of
  // 2048 elements (one sub-batch of 256 threads x 8 bf16)
  const int sub = kScanThreads * 8;
  int want = (1024 + rows - 1) / rows;
  int maxch = (V + sub - 1) / sub;
  int nch = want < 1 ? 1 : (want > maxch ? maxch : want);
  int chunk = (V + nch - 1) / nch;
  chunk = (chunk + sub - 1) / sub * sub;
  g.chunk = chunk;
  g.nchunks = (V + chunk - 1) / chunk;
  return g;
}

size_t scan_bytes(const ScanGeom &g) {
  size_t b = 0;
  const size_t rc = (size_t)g.rows * g.nchunks;
  b += align_up(rc * g.M * sizeof(uint64_t), 256);
  b += align_up(rc * sizeof(float2), 256);
  b += align_up(rc * sizeof(int32_t), 256);
  b += align_up((size_t)g.rows * g.M * sizeof(int32_t), 256);
  b += align_up((size_t)g.rows * g.M * sizeof(float), 256);
  b += align_up((size_t)g.rows * sizeof(float), 256);
  b += align_up((size_t)g.rows * sizeof(int32_t), 256);
  return b;
}

size_t carve_scan(char *base, const ScanGeom &g, Workspace *ws) {
  size_t o = 0;
  const size_t rc = (size_t)g.rows * g.nchunks;
  ws->chunk_keys = reinterpret_cast<uint64_t *>(base + o);
  o += align_up(rc * g.M * sizeof(uint64_t), 256);
  ws->chunk_tail = reinterpret_cast<float2 *>(base + o);
  o += align_up(rc * sizeof(float2), 256);
  ws->chunk_flag = reinterpret_cast<int32_t *>(base + o);
  o += align_up(rc * sizeof(int32_t), 256);
  ws->cand = reinterpret_cast<int32_t *>(base + o);
  o += align_up((size_t)g.rows * g.M * sizeof(int32_t), 256);
  ws->candv = reinterpret_cast<float *>(base + o);
  o += align_up((size_t)g.rows * g.M * sizeof(float), 256);
  ws->tail = reinterpret_cast<float *>(base + o);
  o += align_up((size_t)g.rows * sizeof(float), 256);
  ws->row_flag = reinterpret_cast<int32_t *>(base + o);
  o += align_up((size_t)g.rows * sizeof(int32_t), 256);
  return o;
}

hipError_t launch_scan(const void *logits, int ldt, const ScanGeom &g, float inv_tau,
                       const Workspace &ws, hipStream_t s, hipEvent_t between) {
  const float c = 1.4426950408889634f * inv_tau;  // exp(x / tau) = exp2(x * c)
  dim3 grid(g.nchunks, g.rows);
  const bool aligned = (reinterpret_cast<uintptr_t>(logits) % 16) == 0;
  if (ldt == DT_BF16) {
    const uint16_t *p = static_cast<const uint16_t *>(logits);
    if (aligned && g.V % 8 == 0)
      hipLaunchKernelGGL((scan_chunk_kernel<uint16_t, true>), grid, dim3(kScanThreads), 0, s, p, g,
                         c, ws.chunk_keys, ws.chunk_tail, ws.chunk_flag);
    else
      hipLaunchKernelGGL((scan_chunk_kernel<uint16_t, false>), grid, dim3(kScanThreads), 0, s, p,
                         g, c, ws.chunk_keys, ws.chunk_tail, ws.chunk_flag);
  } else {
    const float *p = static_cast<const float *>(logits);
    if (aligned && g.V % 4 == 0)
      hipLaunchKernelGGL((scan_chunk_kernel<float, true>), grid, dim3(kScanThreads), 0, s, p, g, c,
                         ws.chunk_keys, ws.chunk_tail, ws.chunk_flag);
    else
      hipLaunchKernelGGL((scan_chunk_kernel<float, false>), grid, dim3(kScanThreads), 0, s, p, g,
                         c, ws.chunk_keys, ws.chunk_tail, ws.chunk_flag);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (between) {
    e = hipEventRecord(between, s);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(scan_merge_kernel, dim3(g.rows), dim3(kScanThreads), 0, s, g, c, inv_tau,
                     ws.chunk_keys, ws.chunk_tail, ws.chunk_flag, ws.cand, ws.candv, ws.tail,
                     ws.row_flag);
  return hipGetLastError();
}

}  // namespace dt
