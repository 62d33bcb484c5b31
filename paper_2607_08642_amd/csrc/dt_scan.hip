// S1: per-depth marginal top-M and the tail log-sum-exp (Alg. 1 step 1;
// section 3.2, candidate restriction).
//
// Each logit row [V] is cut into chunks of 10240 elements.  One 256-thread
// workgroup loads its whole chunk into registers (40 values per thread, all
// loads in flight at once) and selects the chunk's M best elements exactly:
//   * keys are 64-bit (order-preserving value bits, ~index), so the order
//     (value desc, id asc) is a plain integer order without ties;
//   * every wave sorts its 64 per-lane maximum keys and takes the ceil(M/4)-th;
//     the minimum over the 4 waves leaves at least M elements at or above it,
//     so it is an exact lower bound on the chunk's M-th best key;
//   * elements below that bound go straight into the running tail sum
//     (max, sum exp((x - max)/tau)); the survivors (about 1% of the chunk on
//     drafter-like rows) are compacted into LDS and bitonic-sorted once; the
//     best M are the chunk's list, the rest join the tail.
// If the survivors overflow the sort buffer (adversarial rows: long runs of
// equal or monotone values), they are streamed through a bounded selector that
// keeps a sorted list of M and flushes a candidate buffer instead.
// The per-row merge (merge_row) sorts the chunk lists of a row together and
// folds the chunk tails; it runs inside the expansion kernel, or in a small
// kernel of its own for dt_scan_topm.
#include "dt_select.h"

namespace dt {

namespace {

using sel::Tail;

constexpr int kWaves = kScanThreads / 64;

struct ScanLDS {
  uint64_t buf[kScanSortCap];
  uint64_t wthr[kWaves];
  float2 red[kWaves];
  int nbuf;
  int nlist;
  int flag;
  uint64_t thr;
};

// ---------------------------------------------------------------------------
// bounded streaming selector (fallback for chunks whose survivors overflow):
// buf[0..nlist) is the sorted best-M list, buf[nlist..nbuf) new candidates
// ---------------------------------------------------------------------------
__device__ void flush(ScanLDS &sh, int M, Tail &tail, float c) {
  const int tid = threadIdx.x;
  const int n = sh.nbuf;
  const int P = sel::pow2_at_least(n, 64);
  for (int i = n + tid; i < P; i += kScanThreads) sh.buf[i] = 0;
  __syncthreads();
  sel::block_sort_desc<kScanThreads>(sh.buf, P);
  for (int i = M + tid; i < n; i += kScanThreads) sel::tail_add1(tail, key_value(sh.buf[i]), c);
  __syncthreads();
  if (tid == 0) {
    const int nl = n < M ? n : M;
    sh.nlist = nl;
    sh.nbuf = nl;
    if (nl == M) {
      const uint64_t t = sh.buf[M - 1] + 1;
      if (t > sh.thr) sh.thr = t;
    }
  }
  __syncthreads();
}

// one group of EPT keys per thread (0 = none); keys below the running
// threshold join the tail, the others the candidate buffer
template <int EPT>
__device__ void stream_batch(ScanLDS &sh, const uint64_t (&key)[EPT], const float (&val)[EPT],
                             int M, Tail &tail, float c) {
  const int lane = threadIdx.x & 63;
  const uint64_t thr = sh.thr;
  float tv[EPT];
  uint64_t bal[EPT];
  int tot = 0;
#pragma unroll
  for (int j = 0; j < EPT; ++j) {
    const bool pass = key[j] != 0 && key[j] >= thr;
    tv[j] = (key[j] != 0 && !pass) ? val[j] : -__builtin_huge_valf();
    bal[j] = __ballot(pass);
    tot += __popcll(bal[j]);
  }
  sel::tail_add_group<EPT>(tail, tv, c);
  if (tot) {
    int base = 0;
    if (lane == 0) base = atomicAdd(&sh.nbuf, tot);
    base = __shfl(base, 0);
    const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
      if ((bal[j] >> lane) & 1ull) sh.buf[base + __popcll(bal[j] & below)] = key[j];
      base += __popcll(bal[j]);
    }
  }
  __syncthreads();
  if (sh.nbuf - sh.nlist > kScanFlushAt) flush(sh, M, tail, c);
}

template <typename T>
struct Elem;
template <>
struct Elem<uint16_t> {
  static constexpr int EPL = 8;  // elements per 16-byte load
};
template <>
struct Elem<float> {
  static constexpr int EPL = 4;
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

// fp32 class test: NaN or +inf (v_cmp_class)
__device__ inline bool nonfinite(float v) { return __builtin_amdgcn_class(v, 0x203); }

// descending bitonic sort of a wave's 64 floats (one per lane)
__device__ inline float wave_sort_desc_f(float v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int k = 2; k <= 64; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const float p = __shfl_xor(v, j);
      const bool desc = (lane & k) == 0;
      const bool lower = (lane & j) == 0;
      v = (desc == lower) ? fmaxf(v, p) : fminf(v, p);
    }
  }
  return v;
}

// inclusive prefix sum over a wave
__device__ inline int wave_incl_scan(int x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  return x;
}

// K1: exact top-M of one chunk (kScanChunk elements) of one row, plus the tail
// of the rest.  Also clears `zero_n` ints at `zero_ptr` (barrier counters of
// the expansion kernel that follows on the stream).
template <typename T, bool VEC>
__global__ __launch_bounds__(kScanThreads) void scan_chunk_kernel(
    const T *__restrict__ logits, ScanGeom g, float c, uint64_t *__restrict__ ckeys,
    float2 *__restrict__ ctail, int32_t *__restrict__ cflag, int32_t *__restrict__ zero_ptr,
    int zero_n) {
  constexpr int EPL = Elem<T>::EPL;
  constexpr int NL = kScanPerThread / EPL;  // 16-byte loads per thread
  constexpr int STEP = kScanThreads * EPL;  // elements per load round
  constexpr float NINF = -__builtin_huge_valf();
  __shared__ ScanLDS sh;
  __shared__ uint64_t list[kMaxM];
  __shared__ float wthr[kWaves];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int row = blockIdx.y, chunk = blockIdx.x;
  const int start = chunk * g.chunk;
  const int n = min(g.chunk, g.V - start);
  const T *base = logits + (size_t)row * g.V + start;
  if (zero_ptr && blockIdx.x == 0 && blockIdx.y == 0)
    for (int i = tid; i < zero_n; i += kScanThreads) zero_ptr[i] = 0;

  // 1. the whole chunk into registers: element (j, e) of this thread has
  //    chunk offset j*STEP + tid*EPL + e; slots past the end hold -inf
  float v[NL][EPL];
#pragma unroll
  for (int j = 0; j < NL; ++j) {
    const int off = j * STEP + tid * EPL;
    if (VEC && off + EPL <= n) {
      if constexpr (EPL == 8) {
        const uint4 r = *reinterpret_cast<const uint4 *>(base + off);
        const uint32_t w4[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          v[j][2 * q] = __uint_as_float(w4[q] << 16);
          v[j][2 * q + 1] = __uint_as_float(w4[q] & 0xFFFF0000u);
        }
      } else {
        const float4 r = *reinterpret_cast<const float4 *>(base + off);
        v[j][0] = r.x;
        v[j][1] = r.y;
        v[j][2] = r.z;
        v[j][3] = r.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < EPL; ++e) v[j][e] = (off + e < n) ? to_f32<T>(base[off + e]) : NINF;
    }
  }
  if (tid == 0) {
    sh.nbuf = 0;
    sh.nlist = 0;
    sh.flag = 0;
  }
  // 2. NaN / +inf flag the row and leave the arithmetic as -inf; thread max
  int bad = 0;
  float tmax = NINF;
#pragma unroll
  for (int j = 0; j < NL; ++j)
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      if (nonfinite(v[j][e])) {
        bad = 1;
        v[j][e] = NINF;
      }
      tmax = fmaxf(tmax, v[j][e]);
    }
  // 3. value threshold: every wave has >= ceil(M/4) lanes whose max is at least
  //    its ceil(M/4)-th largest lane max, so at least M elements of the chunk
  //    are >= the minimum over the waves: no top-M element lies below it
  {
    const float srt = wave_sort_desc_f(tmax);
    const int q = (g.M + kWaves - 1) / kWaves;  // <= 64 since M <= 256
    const float tq = __shfl(srt, q - 1);
    if (lane == 0) wthr[w] = tq;
  }
  __syncthreads();
  float thr = wthr[0];
  for (int i = 1; i < kWaves; ++i) thr = fminf(thr, wthr[i]);
  // 4. count survivors (v >= thr); the others go into this thread's tail, with
  //    the thread max as reference
  Tail tail;
  tail.m = fmaxf(tmax, -3.402823466e38f);
  float s = 0.0f;
  int cnt = 0;
#pragma unroll
  for (int j = 0; j < NL; ++j)
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      const int off = j * STEP + tid * EPL + e;
      const bool in = off < n;
      const bool pass = in && v[j][e] >= thr;
      cnt += pass;
      const float ex = exp2f((v[j][e] - tail.m) * c);
      s += (in && !pass) ? ex : 0.0f;
    }
  tail.s = s;
  if (bad) atomicOr(&sh.flag, 1);
  // 5. survivor slots: wave prefix of the per-thread counts, one LDS atomic per wave
  const int incl = wave_incl_scan(cnt);
  int wbase = 0;
  if (lane == 63 && incl) wbase = atomicAdd(&sh.nbuf, incl);
  wbase = __shfl(wbase, 63);
  __syncthreads();
  const int nsurv = sh.nbuf;
  const int M = g.M;
  if (nsurv <= kScanSortCap) {
    int pos = wbase + incl - cnt;
    if (cnt) {
#pragma unroll
      for (int j = 0; j < NL; ++j)
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
          const int off = j * STEP + tid * EPL + e;
          if (off < n && v[j][e] >= thr) sh.buf[pos++] = make_key(v[j][e], (uint32_t)(start + off));
        }
    }
    __syncthreads();
    if (nsurv <= 2 * kScanThreads) {
      // 6a. rank sort: each survivor's rank is the number of larger keys
      for (int i = tid; i < M; i += kScanThreads) list[i] = 0ull;
      __syncthreads();
      for (int i = tid; i < nsurv; i += kScanThreads) {
        const uint64_t k = sh.buf[i];
        int rank = 0;
        for (int q = 0; q < nsurv; ++q) rank += sh.buf[q] > k;
        if (rank < M)
          list[rank] = k;
        else
          sel::tail_add1(tail, key_value(k), c);
      }
      if (tid == 0) sh.nlist = nsurv < M ? nsurv : M;
      __syncthreads();
    } else {
      // 6b. bitonic sort of the survivors
      const int P = sel::pow2_at_least(nsurv, 64);
      for (int i = nsurv + tid; i < P; i += kScanThreads) sh.buf[i] = 0;
      __syncthreads();
      sel::block_sort_desc<kScanThreads>(sh.buf, P);
      for (int i = M + tid; i < nsurv; i += kScanThreads) sel::tail_add1(tail, key_value(sh.buf[i]), c);
      for (int i = tid; i < M; i += kScanThreads) list[i] = i < nsurv ? sh.buf[i] : 0ull;
      if (tid == 0) sh.nlist = nsurv < M ? nsurv : M;
      __syncthreads();
    }
  } else {
    // 6c. fallback (adversarial rows): stream the survivors through the
    //     bounded selector, starting from the value threshold
    __syncthreads();
    if (tid == 0) {
      sh.nbuf = 0;
      sh.nlist = 0;
      sh.thr = 1;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NL; ++j) {
      uint64_t key[EPL];
      float val[EPL];
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const int off = j * STEP + tid * EPL + e;
        key[e] = (off < n && v[j][e] >= thr) ? make_key(v[j][e], (uint32_t)(start + off)) : 0ull;
        val[e] = v[j][e];
      }
      stream_batch<EPL>(sh, key, val, M, tail, c);
    }
    if (sh.nbuf > sh.nlist) flush(sh, M, tail, c);
    for (int i = tid; i < M; i += kScanThreads) list[i] = i < sh.nlist ? sh.buf[i] : 0ull;
    __syncthreads();
  }
  const Tail t = sel::block_tail<kScanThreads>(tail, c, sh.red);
  const size_t cidx = (size_t)row * g.nchunks + chunk;
  uint64_t *out = ckeys + cidx * M;
  for (int i = tid; i < M; i += kScanThreads) out[i] = list[i];
  if (tid == 0) {
    ctail[cidx] = make_float2(t.m, t.s);
    cflag[cidx] = sh.flag ? DT_TREE_NONFINITE : 0;
  }
}

// K2 (dt_scan_topm only): merge the chunk lists of one row
__global__ __launch_bounds__(kScanThreads) void scan_merge_kernel(
    ScanGeom g, float c, float inv_tau, const uint64_t *__restrict__ ckeys,
    const float2 *__restrict__ ctail, const int32_t *__restrict__ cflag, int32_t *__restrict__ cand,
    float *__restrict__ candv, float *__restrict__ tailR, int32_t *__restrict__ rflag) {
  extern __shared__ uint64_t sortbuf[];  // merge_buf_bytes(nchunks, M)
  __shared__ float2 red[kWaves];
  __shared__ int flag;
  const int row = blockIdx.x;
  sel::merge_row<kScanThreads, false>(ckeys + (size_t)row * g.nchunks * g.M, g.nchunks, g.M,
                                      ctail + (size_t)row * g.nchunks, cflag + (size_t)row * g.nchunks,
                                      c, inv_tau, sortbuf, red, &flag, cand + (size_t)row * g.M,
                                      candv + (size_t)row * g.M, tailR + row, rflag + row,
                                      nullptr);
}

}  // namespace

ScanGeom scan_geom(int rows, int V, int M) {
  ScanGeom g;
  g.rows = rows;
  g.V = V;
  g.M = M;
  g.chunk = kScanChunk;
  g.nchunks = (V + kScanChunk - 1) / kScanChunk;
  return g;
}

size_t merge_lds_bytes(const ScanGeom &g) { return (size_t)sel::merge_buf_bytes(g.nchunks, g.M); }

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

hipError_t launch_scan_chunks(const void *logits, int ldt, const ScanGeom &g, float inv_tau,
                              const Workspace &ws, int32_t *zero_ptr, int zero_n, hipStream_t s) {
  const float c = 1.4426950408889634f * inv_tau;  // exp(x / tau) = exp2(x * c)
  dim3 grid(g.nchunks, g.rows);
  const bool aligned = (reinterpret_cast<uintptr_t>(logits) % 16) == 0;
  if (ldt == DT_BF16) {
    const uint16_t *p = static_cast<const uint16_t *>(logits);
    if (aligned && g.V % 8 == 0)
      hipLaunchKernelGGL((scan_chunk_kernel<uint16_t, true>), grid, dim3(kScanThreads), 0, s, p, g,
                         c, ws.chunk_keys, ws.chunk_tail, ws.chunk_flag, zero_ptr, zero_n);
    else
      hipLaunchKernelGGL((scan_chunk_kernel<uint16_t, false>), grid, dim3(kScanThreads), 0, s, p,
                         g, c, ws.chunk_keys, ws.chunk_tail, ws.chunk_flag, zero_ptr, zero_n);
  } else {
    const float *p = static_cast<const float *>(logits);
    if (aligned && g.V % 4 == 0)
      hipLaunchKernelGGL((scan_chunk_kernel<float, true>), grid, dim3(kScanThreads), 0, s, p, g, c,
                         ws.chunk_keys, ws.chunk_tail, ws.chunk_flag, zero_ptr, zero_n);
    else
      hipLaunchKernelGGL((scan_chunk_kernel<float, false>), grid, dim3(kScanThreads), 0, s, p, g,
                         c, ws.chunk_keys, ws.chunk_tail, ws.chunk_flag, zero_ptr, zero_n);
  }
  return hipGetLastError();
}

hipError_t launch_scan_merge(const ScanGeom &g, float inv_tau, const Workspace &ws, hipStream_t s) {
  const float c = 1.4426950408889634f * inv_tau;
  const size_t lds = merge_lds_bytes(g);
  hipError_t e = hipFuncSetAttribute((const void *)scan_merge_kernel,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(scan_merge_kernel, dim3(g.rows), dim3(kScanThreads), lds, s, g, c, inv_tau,
                     ws.chunk_keys, ws.chunk_tail, ws.chunk_flag, ws.cand, ws.candv, ws.tail,
                     ws.row_flag);
  return hipGetLastError();
}

}  // namespace dt
