// S1: per-depth marginal top-M and the tail log-sum-exp (Alg. 1 step 1;
// section 3.2, candidate restriction).
//
// Each logit row [V] is cut into segments of one or more batches of 10240
// elements; a 256-thread workgroup streams its segment's batches through
// registers (40 values per thread, the next batch always in flight) against a
// running exact top-M list:
//   * keys are 64-bit (order-preserving value bits, ~index), so the order
//     (value desc, id asc) is a plain integer order without ties;
//   * first batch: every wave finds the ceil(M/4)-th largest of its 64 per-lane
//     maxima (a bitwise search with one ballot per bit); the minimum over the
//     4 waves leaves at least M elements at or above it, so it is an exact
//     lower bound on the batch's M-th best element;  later batches: the list's
//     M-th value;
//   * one pass over the registers sends every element below that threshold
//     into the running tail sum (max, sum exp((x - max)/tau)); the few above
//     it are appended, as keys, to a per-wave region of LDS through the
//     comparison's lane mask;
//   * the regions are merged into the list after the first batch, once about
//     2M candidates have gathered, and at the end.  For M <= 64 each wave
//     sorts its region in registers (bitonic, 64 keys per lane-set) and the
//     wave lists and the list meet in a tree of bitonic merges; larger M ranks
//     every candidate by counting the larger ones (or sorts when there are
//     many).  Keys that drop out of the list join the tail.
// If a wave's candidates overflow its region (adversarial rows: long runs of
// equal or monotone values), the batch is streamed through a bounded selector
// that keeps a sorted list of M.
// The per-row merge of the segment lists (merge_row and its register
// variants) runs inside the expansion kernel, or in a small kernel of its own
// for dt_scan_topm.
//
// For Domino's own head the launch carries extra workgroups (blockIdx.x >=
// nchunks) that compute a[row][r] = W_1^H H_row, the half of W_1 [H_d; S] that
// does not depend on the path (section 2.3): a small GEMM of 16 x 16 MFMA
// tiles whose memory time hides under the scan's.
#include "dt_select.h"
#include <hip/hip_ext.h>

#include <type_traits>

namespace dt {

namespace {

using sel::Tail;

constexpr int kWaves = kScanThreads / 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// One 16-rank x 16-row tile of a = W_1^H H (tile = rank tile + (rank tiles) x
// row tile) with fp32 accumulation: the K = d_H columns split over the waves
// in chunks of KC (one MFMA group: lane l holds KC/4 consecutive columns of
// rank (tile row) l % 16 and of H row l % 16, at column group l / 16), the
// wave partials summed in LDS (red: kWaves x 256 floats).  Out-of-range ranks,
// rows and columns read as zeros and are not stored.  bf16: 16x16x32 bf16
// MFMAs on the stored values (exact products); fp32: 16x16x4 fp32 MFMAs.
template <typename TW>
__device__ void head_proj_tile(const HeadProj &p, int rows, int tile, float *red) {
  const int nrt = (p.rank + 15) / 16;
  if (tile >= nrt * ((rows + 15) / 16)) return;  // (whole workgroup)
  const int rt = tile % nrt, qt = tile / nrt;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4;
  const int r = rt * 16 + (lane & 15), q = qt * 16 + (lane & 15);
  const bool rok = r < p.rank, qok = q < rows;
  const TW *wr = static_cast<const TW *>(p.w1) + (size_t)(rok ? r : 0) * p.ld1;
  const TW *hr = static_cast<const TW *>(p.H) + (size_t)(qok ? q : 0) * p.d_H;
  constexpr bool kBf = sizeof(TW) == 2;
  constexpr int KC = kBf ? 32 : 16, KL = KC / 4;  // columns per chunk, per lane
  constexpr int U = 4;                             // chunks in flight per wave
  using V = typename std::conditional<kBf, uint4, float4>::type;  // KL columns
  const int nch = (p.d_H + KC - 1) / KC;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int c0 = w; c0 < nch; c0 += kWaves * U) {
    V av[U], bv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = (c0 + u * kWaves) * KC + g * KL;  // (d_H % 8 == 0: a lane's KL are all in or out)
      const bool ok = c0 + u * kWaves < nch && k < p.d_H;
      av[u] = (ok && rok) ? *reinterpret_cast<const V *>(wr + k) : V{};
      bv[u] = (ok && qok) ? *reinterpret_cast<const V *>(hr + k) : V{};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if constexpr (kBf) {
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, av[u]),
                                                     __builtin_bit_cast(bf16x8, bv[u]), acc, 0, 0, 0);
      } else {
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u].x, bv[u].x, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u].y, bv[u].y, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u].z, bv[u].z, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u].w, bv[u].w, acc, 0, 0, 0);
      }
    }
  }
  // lane l, register i: rank rt*16 + (l/16)*4 + i, row qt*16 + l%16
#pragma unroll
  for (int i = 0; i < 4; ++i) red[w * 256 + lane * 4 + i] = acc[i];
  __syncthreads();
  static_assert(kScanThreads == 256, "one thread per tile element");
  const int e = threadIdx.x, el = e >> 2, ei = e & 3;
  float sum = red[e];
  for (int v = 1; v < kWaves; ++v) sum += red[v * 256 + e];
  const int rr = rt * 16 + (el >> 4) * 4 + ei, qq = qt * 16 + (el & 15);
  if (rr < p.rank && qq < rows) p.a[(size_t)qq * p.rank + rr] = sum;
}

constexpr int kRegion = kScanSortCap / kWaves;       // candidate keys per wave
constexpr int kRegionCap = kRegion - kMaxM / kWaves;  // fill limit: the list fits beside them
// a merge is due once this many times M candidates have gathered (measured best
// at 2 for Qwen3 shapes: 1, 4 and 8 were slower)
constexpr int kMergeAt = 2;

struct ScanLDS {
  alignas(16) uint64_t buf[kScanSortCap];
  float2 red[kWaves];
  // per-wave candidate counts, by batch parity: a wave can start the next batch
  // (and write its counts) while another still reads this batch's
  int wcnt[2][kWaves];
  int wprev[2][kWaves];
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

// The bitwise search for a bound runs down to this bit: a bf16 value's
// order-preserving code is set by its high 16 bits (its low 16 are 0 for a
// value >= 0 and all ones below 0), so 16 steps of one ballot each (a serial
// chain) find the high half of the q-th largest code, and full_code restores
// the low half.
template <typename T>
constexpr int kLowBit = 0;
template <>
constexpr int kLowBit<uint16_t> = 16;
template <typename T>
__device__ inline uint32_t full_code(uint32_t pre) {
  if constexpr (kLowBit<T> == 16) return (pre & 0x80000000u) ? pre : (pre | 0xFFFFu);
  return pre;
}

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

// Raw registers of one batch: kScanPerThread elements per thread as 16-byte loads
template <typename T>
struct Raw {
  static constexpr int NL = kScanPerThread / Elem<T>::EPL;
  uint4 q[NL];
};

// Issue the loads of one batch (element (j, e) of this thread sits at batch
// offset j*STEP + tid*EPL + e); nothing waits for them here.
template <typename T, bool VEC>
__device__ inline void load_batch(Raw<T> &r, const T *base, int bn) {
  constexpr int EPL = Elem<T>::EPL;
  constexpr int STEP = kScanThreads * EPL;
  int lb = threadIdx.x * EPL;
  asm volatile("" : "+v"(lb));
#pragma unroll
  for (int j = 0; j < Raw<T>::NL; ++j) {
    const int off = lb + j * STEP;
    if (VEC && off + EPL <= bn) {
      r.q[j] = *reinterpret_cast<const uint4 *>(base + off);
    } else {
      uint32_t w[4] = {0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u};  // bf16 -inf pairs
      if constexpr (EPL == 8) {
        const uint16_t *b16 = reinterpret_cast<const uint16_t *>(base);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t h = off + e < bn ? (uint32_t)b16[off + e] : 0xFF80u;
          w[e >> 1] = (e & 1) ? ((w[e >> 1] & 0xFFFFu) | (h << 16)) : ((w[e >> 1] & 0xFFFF0000u) | h);
        }
      } else {
        const float *f = reinterpret_cast<const float *>(base);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          w[e] = __float_as_uint(off + e < bn ? f[off + e] : -__builtin_huge_valf());
      }
      r.q[j] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

// 16-byte-aligned rows: straight-line buffer loads of batch `b` of a segment
// (seg_bytes of data from `seg`); loads past the segment's end return zeros
// (each 16-byte load lies wholly inside or outside it) and are made -inf by
// pad_batch.  Nothing waits for the data here.
template <typename T>
__device__ inline void load_batch_vec(Raw<T> &r, __amdgpu_buffer_rsrc_t seg, int b) {
  constexpr int EPL = Elem<T>::EPL;
  constexpr int STEP = kScanThreads * EPL;
  int lb = (int)threadIdx.x * EPL;
  asm volatile("" : "+v"(lb));
  const int base = (b * kScanChunk + lb) * (int)sizeof(T);
#pragma unroll
  for (int j = 0; j < Raw<T>::NL; ++j)
    r.q[j] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                           seg, base + j * STEP * (int)sizeof(T), 0, 0));
}

// the elements of a partial batch past its end become -inf
template <typename T>
__device__ inline void pad_batch(Raw<T> &r, int bn) {
  constexpr int EPL = Elem<T>::EPL;
  constexpr int STEP = kScanThreads * EPL;
  const uint32_t ninf = EPL == 8 ? 0xFF80FF80u : 0xFF800000u;
#pragma unroll
  for (int j = 0; j < Raw<T>::NL; ++j)
    if ((int)threadIdx.x * EPL + j * STEP >= bn) r.q[j] = make_uint4(ninf, ninf, ninf, ninf);
}

// Opaque to the compiler: each pass unpacks the elements again (one ALU op each)
// instead of keeping every unpacked value live across the passes.
template <typename T>
__device__ inline void fence_regs(Raw<T> &r) {
#pragma unroll
  for (int j = 0; j < Raw<T>::NL; ++j) asm volatile("" : "+v"(r.q[j].x), "+v"(r.q[j].y), "+v"(r.q[j].z), "+v"(r.q[j].w));
}

// element e of 16-byte load j (unpacked from the raw registers on each use)
template <typename T>
__device__ inline float elem(const Raw<T> &r, int j, int e) {
  const uint4 q = r.q[j];
  if constexpr (Elem<T>::EPL == 8) {
    const uint32_t wd = (e >> 1) == 0 ? q.x : (e >> 1) == 1 ? q.y : (e >> 1) == 2 ? q.z : q.w;
    return (e & 1) ? __uint_as_float(wd & 0xFFFF0000u) : __uint_as_float(wd << 16);
  } else {
    return __uint_as_float(e == 0 ? q.x : e == 1 ? q.y : e == 2 ? q.z : q.w);
  }
}

// K1: exact top-M of one segment (g.chunk elements: one or more batches of
// kScanChunk) of one row, plus the tail of the rest.  The segment's batches
// stream through registers (the next batch loads while this one is processed)
// against a running top-M list:
//   first batch  the value threshold above, then a rank pass;
//   later ones   only elements above the list's M-th value can enter (later
//                elements lose ties on the index); they are ranked into the list
//                and whatever drops out joins the tail.
// The tail of the elements below the threshold is summed against `ref`, the
// largest value seen so far (never below them, so nothing overflows).
// Also clears `zero_n` ints at `zero_ptr` (barrier counters of the expansion
// kernel that follows on the stream).
// TWP: the weights dtype of a head projection carried by the launch (void: none)
template <typename T, bool VEC, typename TWP = void>
__global__ __launch_bounds__(kScanThreads) void scan_chunk_kernel(
    const T *__restrict__ logits, ScanGeom g, float c, uint64_t *__restrict__ ckeys,
    float2 *__restrict__ ctail, int32_t *__restrict__ cflag, int32_t *__restrict__ zero_ptr,
    int zero_n, HeadProj hp) {
  constexpr int EPL = Elem<T>::EPL;
  constexpr int NL = Raw<T>::NL;
  constexpr int STEP = kScanThreads * EPL;
  constexpr float NINF = -__builtin_huge_valf();
  __shared__ ScanLDS sh;
  __shared__ uint64_t list[2][kMaxM];
  __shared__ float wthr[kWaves];
  if constexpr (!std::is_void<TWP>::value) {
    if ((int)blockIdx.x >= g.nchunks) {
      head_proj_tile<TWP>(hp, g.rows, blockIdx.y * hp.extra + blockIdx.x - g.nchunks,
                          reinterpret_cast<float *>(sh.buf));
      return;
    }
  }
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int row = blockIdx.y, seg = blockIdx.x;
  const int M = g.M;
  const int seg_start = seg * g.chunk;
  const int seg_n = min(g.chunk, g.V - seg_start);
  const int nbat = (seg_n + kScanChunk - 1) / kScanChunk;
  const T *rowp = logits + (size_t)row * g.V + seg_start;
  if (zero_ptr && blockIdx.x == 0 && blockIdx.y == 0)
    for (int i = tid; i < zero_n; i += kScanThreads) zero_ptr[i] = 0;

  Raw<T> ra, rb;
  const __amdgpu_buffer_rsrc_t segr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<T *>(rowp), 0, seg_n * (int)sizeof(T), 0x00020000);
  auto load = [&](Raw<T> &r, int b) {
    if constexpr (VEC)
      load_batch_vec<T>(r, segr, b);
    else
      load_batch<T, false>(r, rowp + (size_t)b * kScanChunk, min(kScanChunk, seg_n - b * kScanChunk));
  };
  load(ra, 0);
  if (tid == 0) sh.flag = 0;
  for (int i = tid; i < M; i += kScanThreads) list[0][i] = 0ull;

  int cur = 0, nl = 0;    // running list: list[cur][0..nl), sorted descending
  float thr = NINF;       // after the first merge: only values above thr can enter
  int wbase = 0;          // candidates of this wave since the last merge
  Tail tail = sel::tail_empty();

  // Merge the candidates in the regions (wc[r] keys each, all >= the list's
  // threshold) into the running list; the keys that drop out join the tail.
  auto merge_regions = [&](const int (&wc)[kWaves]) {
    int nc = 0;
#pragma unroll
    for (int i = 0; i < kWaves; ++i) nc += wc[i];
    if (nc == 0) return;
    const uint64_t *L0 = list[cur];
    uint64_t *L1 = list[cur ^ 1];
    if (M <= 64) {
      // In registers: every wave sorts its own region (chunks of 64, even waves
      // descending, odd ones ascending), keeping its best 64; the four lists
      // and then the running list meet in a tree (sel::merge_halves).  Every
      // key that drops out joins this lane's tail.
      static_assert(kWaves == 4, "merge tree of four waves");
      const bool mydesc = (w & 1) == 0;
      uint64_t *rg = sh.buf + w * kRegion;
      const int n = wc[w];
      uint64_t v = sel::wave_sort64(lane < n ? rg[lane] : 0ull, mydesc);
      for (int c0 = 64; c0 < n; c0 += 64) {
        const uint64_t ch = sel::wave_sort64(c0 + lane < n ? rg[c0 + lane] : 0ull, !mydesc);
        v = mydesc ? sel::merge_halves(v, ch, true, tail, c) : sel::merge_halves(ch, v, false, tail, c);
      }
      if (w & 1) rg[lane] = v;  // (a wave only ever reads its own region before this)
      __syncthreads();
      if ((w & 1) == 0) {
        v = sel::merge_halves(v, sh.buf[(w + 1) * kRegion + lane], w == 0, tail, c);
        if (w == 2) rg[lane] = v;
      }
      __syncthreads();
      if (w == 0) {
        v = sel::merge_halves(v, sh.buf[2 * kRegion + lane], true, tail, c);
        const int li = 63 - lane;  // the running list, reversed
        v = sel::merge_halves(v, li < nl ? L0[li] : 0ull, true, tail, c);
        if (lane >= M && v) sel::tail_add1(tail, key_value(v), c);
        if (lane < M) L1[lane] = v;
      }
    } else {
#pragma unroll
    for (int i = 0; i < kWaves; ++i)
      if (tid == i && (wc[i] & 1)) sh.buf[i * kRegion + wc[i]] = 0ull;  // pad for paired reads
    __syncthreads();
    if (nc + nl <= 4 * kScanThreads) {
      // a candidate's rank is the number of larger candidates (paired reads
      // over the regions) plus the number of larger list keys (binary search);
      // a list key's rank is its position plus the number of larger candidates
      for (int it = tid; it < nc + nl; it += kScanThreads) {
        uint64_t k;
        int rank;
        if (it < nc) {
          int r = 0, o = it;
#pragma unroll
          for (int i = 0; i < kWaves - 1; ++i)
            if (r == i && o >= wc[i]) {
              o -= wc[i];
              r = i + 1;
            }
          k = sh.buf[r * kRegion + o];
          int lo = 0, hi = nl;
          while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (L0[mid] > k)
              lo = mid + 1;
            else
              hi = mid;
          }
          rank = lo;
        } else {
          rank = it - nc;
          k = L0[rank];
        }
#pragma unroll
        for (int r2 = 0; r2 < kWaves; ++r2) {
          const ulonglong2 *p2 = reinterpret_cast<const ulonglong2 *>(sh.buf + r2 * kRegion);
          const int np = (wc[r2] + 1) >> 1;
#pragma unroll 4
          for (int i = 0; i < np; ++i) {
            const ulonglong2 kk = p2[i];
            rank += (kk.x > k) + (kk.y > k);
          }
        }
        if (rank < M)
          L1[rank] = k;
        else
          sel::tail_add1(tail, key_value(k), c);
      }
    } else {
      // many candidates: clear the unused part of every region, put the list
      // keys into the free slots (the regions never fill past kRegionCap, so
      // they fit), sort everything
      for (int r = 0; r < kWaves; ++r)
        for (int i = wc[r] + tid; i < kRegion; i += kScanThreads) sh.buf[r * kRegion + i] = 0ull;
      __syncthreads();
      for (int i = tid; i < nl; i += kScanThreads) {
        int r = 0, o = i;
#pragma unroll
        for (int x = 0; x < kWaves - 1; ++x)
          if (r == x && o >= kRegion - wc[x]) {
            o -= kRegion - wc[x];
            r = x + 1;
          }
        sh.buf[r * kRegion + wc[r] + o] = L0[i];
      }
      __syncthreads();
      sel::block_sort_desc<kScanThreads>(sh.buf, kScanSortCap);
      const int tot = nc + nl;
      for (int i = M + tid; i < tot; i += kScanThreads) sel::tail_add1(tail, key_value(sh.buf[i]), c);
      for (int i = tid; i < M; i += kScanThreads) L1[i] = i < tot ? sh.buf[i] : 0ull;
    }
    }
    __syncthreads();
    cur ^= 1;
    nl = nc + nl < M ? nc + nl : M;
  };

  // after a merge: the threshold and the tail reference follow the list's M-th
  // value (later tail elements lie at or below it)
  auto after_merge = [&]() {
    if (nl == M) thr = fmaxf(thr, key_value(list[cur][M - 1]));
    if (thr > tail.m) {
      tail.s *= sel::fast_exp2((tail.m - thr) * c);
      tail.m = thr;
    }
    wbase = 0;
  };

  // one batch: b = batch index in the segment, raw = its registers.  The
  // candidates accumulate in the regions; they are merged after the first
  // batch (which sets the threshold), once about 2M have gathered (each merge
  // raises the threshold), and at the end.
  auto process = [&](Raw<T> &raw, int b) {
    const int bstart = b * kScanChunk;
    const int bn = min(kScanChunk, seg_n - bstart);
    const bool first = b == 0;
    if (VEC && bn < kScanChunk) pad_batch<T>(raw, bn);
    // this thread's first element offset, opaque so that the per-element
    // offsets are formed at each use rather than hoisted (40 registers)
    int lb = tid * EPL;
    asm volatile("" : "+v"(lb));
    if (first) {
      // every wave has >= q = ceil(M/4) lanes whose max is at least its q-th
      // largest lane max, so at least M elements of the batch are >= the
      // minimum over the waves: no top-M element lies below it.  The q-th
      // largest is found bit by bit on order-preserving codes, one ballot per bit.
      float tmax = NINF;
#pragma unroll
      for (int j = 0; j < NL; ++j)
#pragma unroll
        for (int e = 0; e < EPL; ++e) tmax = fmaxf(tmax, elem<T>(raw, j, e));
      const int q = (M + kWaves - 1) / kWaves;  // <= 64 since M <= 256
      const uint32_t code = ordered_bits(tmax);
      uint32_t pre = 0;
#pragma unroll
      for (int bit = 31; bit >= kLowBit<T>; --bit) {
        const uint32_t cand = pre | (1u << bit);
        if (__popcll(__ballot(code >= cand)) >= q) pre = cand;
      }
      pre = full_code<T>(pre);
      if (lane == 0) wthr[w] = ordered_to_float(pre);
      __syncthreads();
      thr = wthr[0];
#pragma unroll
      for (int i = 1; i < kWaves; ++i) thr = fminf(thr, wthr[i]);
      // (the tail's reference follows the threshold, at or above every element
      // the tail takes, not the maximum: see the wave kernel)
      tail.m = fmaxf(thr, -3.402823466e38f);
    }
    // Candidate test: the first batch keeps ties with its lower bound; later
    // elements must beat the list's M-th value (they lose ties on the index).
    // With a lower bound of -inf (fewer than M finite elements) the first
    // batch keeps everything in range.
    const float tb = thr;
    const bool all_in = first && !(tb > NINF);
    // One pass over the registers: the tail of the elements that cannot enter
    // (against tail.m, which is >= all of them) and, for the rare elements that
    // can, their key appended to this wave's region (wave-uniform branch on the
    // comparison's lane mask; order (element, lane)).
    fence_regs<T>(raw);
    // one comparison x > te: te = tb for later batches; for the first batch
    // any value below tb does (a few extra candidates are ranked exactly)
    const float te = first && tb > NINF ? tb - (fabsf(tb) * 0x1p-20f + 0x1p-126f) : tb;
    uint64_t *region = sh.buf + w * kRegion;
    int wpos = wbase;  // wave-uniform
    auto append = [&](bool pass, float x, int off) {
      const uint64_t bal = __ballot(pass);
      if (bal) {
        const int at = wpos + __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                        __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0));
        if (pass && at < kRegionCap) region[at] = make_key(x, (uint32_t)(seg_start + bstart + off));
        wpos += __popcll(bal);
      }
    };
    // exp((x - m) / tau) = 2^((x - m) c), 0 for candidates and padding.  While
    // |m c| <= 128 the exponent is one fma, x c - (m c), off by at most half an
    // ulp of m c (2^-17, the same for every term); otherwise two operations.
    auto tail_pass = [&](auto expo) {
      float s = 0.0f;
#pragma unroll
      for (int j = 0; j < NL; ++j)
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
          const float x = elem<T>(raw, j, e);
          const bool pass = x > te;
          s += sel::fast_exp2(pass ? NINF : expo(x));
          append(pass, x, lb + j * STEP + e);
        }
      tail.s += s;
    };
    {
      const float m = tail.m, mc = m * c;
      if (fabsf(mc) <= 128.0f)
        tail_pass([=](float x) { return __builtin_fmaf(x, c, -mc); });
      else
        tail_pass([=](float x) { return (x - m) * c; });
    }
    if (all_in) {
      // a lower bound of -inf: the -inf elements in range are candidates too
      // (read again from memory; the tail pass gave them nothing)
#pragma unroll 1
      for (int k = 0; k < NL * EPL; ++k) {
        const int off = lb + (k / EPL) * STEP + k % EPL;
        append(off < bn && to_f32<T>(rowp[bstart + off]) == NINF, NINF, off);
      }
    }
    const int wn = wpos - wbase;
    // the same candidate set, element by element (used by the fallback below)
    auto is_cand = [&](float x, int off) { return x > te || (all_in && off < bn && x == NINF); };
    const int wprev = wbase;
    wbase += wn;
    const int par = b & 1;
    if (lane == 0) {
      sh.wcnt[par][w] = wbase;
      sh.wprev[par][w] = wprev;
    }
    __syncthreads();
    int wc[kWaves], wp[kWaves];
    bool overflow = false, crowded = false;
    int ncand = 0;
#pragma unroll
    for (int i = 0; i < kWaves; ++i) {
      wc[i] = sh.wcnt[par][i];
      wp[i] = sh.wprev[par][i];
      overflow |= wc[i] > kRegionCap;
      crowded |= wc[i] > kRegionCap / 2;
      ncand += wc[i];
    }
    if (!overflow) {
      // a merge costs a fixed latency plus a term growing with the candidates
      if (first || crowded || ncand >= kMergeAt * M || b == nbat - 1) {
        merge_regions(wc);
        after_merge();
      }
      return;
    }
    // a region overflowed (adversarial rows): merge what the earlier batches
    // left, then stream this batch's candidates through the bounded selector,
    // starting from the list
    merge_regions(wp);
    after_merge();
    const uint64_t *L0 = list[cur];
    uint64_t *L1 = list[cur ^ 1];
    for (int i = tid; i < nl; i += kScanThreads) sh.buf[i] = L0[i];
    if (tid == 0) {
      sh.nbuf = nl;
      sh.nlist = nl;
      sh.thr = nl == M ? L0[M - 1] + 1 : 1ull;
    }
    __syncthreads();
    // (the batch is read again from memory, one load group at a time)
#pragma unroll 1
    for (int j = 0; j < NL; ++j) {
      uint64_t key[EPL];
      float val[EPL];
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const int off = lb + j * STEP + e;
        const float x = off < bn ? to_f32<T>(rowp[bstart + off]) : NINF;
        const bool pass = is_cand(x, off);
        key[e] = pass ? make_key(x, (uint32_t)(seg_start + bstart + off)) : 0ull;
        val[e] = pass ? x : NINF;  // the non-candidates are already in the tail
      }
      stream_batch<EPL>(sh, key, val, M, tail, c);
    }
    if (sh.nbuf > sh.nlist) flush(sh, M, tail, c);
    const int nn = sh.nlist;
    for (int i = tid; i < M; i += kScanThreads) L1[i] = i < nn ? sh.buf[i] : 0ull;
    __syncthreads();
    cur ^= 1;
    nl = nn;
    after_merge();
  };

  // the next batch is always in flight while one is processed; VEC loads past
  // the segment's end return zeros and cost no memory traffic
  for (int b = 0; b < nbat; b += 2) {
    if (VEC || b + 1 < nbat) load(rb, b + 1);
    process(ra, b);
    if (VEC || b + 2 < nbat) load(ra, b + 2);
    if (b + 1 < nbat) process(rb, b + 1);
  }

  // a NaN makes a tail sum NaN (it never passes a comparison); +inf heads the list
  if (!(tail.s == tail.s) || (nl && key_value(list[cur][0]) == __builtin_huge_valf()))
    atomicOr(&sh.flag, 1);
  const Tail t = sel::block_tail<kScanThreads>(tail, c, sh.red);
  const size_t cidx = (size_t)row * g.nchunks + seg;
  uint64_t *out = ckeys + cidx * M;
  for (int i = tid; i < M; i += kScanThreads) out[i] = i < nl ? list[cur][i] : 0ull;
  if (tid == 0) {
    ctail[cidx] = make_float2(t.m, t.s);
    cflag[cidx] = sh.flag ? DT_TREE_NONFINITE : 0;
  }
}

// ---------------------------------------------------------------------------
// Wave-streaming variant (M <= 64, rows read with 16-byte loads): the same
// segments, batches and per-element work, but each wave keeps its own list of
// its 64 best keys in registers (lane p: position p, descending) and merges
// its own candidates into it when they gather -- no block barrier while the
// segment streams, so a wave that merges does not hold up the other waves'
// loads.  A candidate must beat a lower bound on the segment's M-th key:
//   * the bound tb of the first two batches (as above, over the lane maxima of
//     both; the one block barrier), ties kept.  Drawn from twice the elements,
//     it admits about 40% fewer candidates over an eight-batch segment of
//     Gaussian-like logits than the first batch's alone;
//   * the wave's own list's M-th value, strictly: the wave's later elements
//     have larger indices, so they lose ties with its own list.
// Both depend on nothing but the data, so the candidates, the merges and the
// order of every tail sum are the same from run to run.  (Reading the other
// waves' list values as they stood was faster -- 40.2 against 43.3 us on 512
// rows of 151936 bf16 logits -- but made the candidates, and with them the
// tails' rounding, depend on timing; reading them two batches late, waiting
// for them, gained nothing over the own bound.)
// A wave merges once 48 candidates have gathered (fewer merges than at 32,
// with the bound from two batches rising early enough).  The region holds
// (index, value bits) pairs; the keys are formed in the merge.
// The four wave lists meet once, at the end of the segment (two pairs side by
// side, then the two results).  A wave whose
// candidates overflow its region re-reads the batch and merges as it goes;
// a first batch without a finite bound (mostly -inf or padding) takes every
// element in range as a candidate that way.
// Each wave keeps its next batch in flight in registers (two buffers; a third,
// two batches ahead, measured slower: 43.2 against 40.0 us on 512 rows of
// 151936 bf16 logits, with the bounds shared), four workgroups per CU.
// ---------------------------------------------------------------------------
template <typename T>
struct WaveScan {
  static constexpr int kBufs = 2;  // register batches per thread (2 or 3)
  static constexpr int kRegion = 512;  // candidate keys a wave gathers between merges
};

// merge region[0..n) ((index << 32) | value bits each) into the wave's list
// (descending keys, one per lane); keys that fall out of the best 64 join the
// lane's tail.  fresh: the list is still empty, and the first 64 keys become
// it sorted, with nothing to merge (wave-uniform; cleared here).
__device__ inline void wave_merge(const uint64_t *region, int n, uint64_t &list, bool &fresh, Tail &tail,
                                  float c) {
  const int lane = threadIdx.x & 63;
  for (int c0 = 0; c0 < n; c0 += 64) {
    uint64_t k = 0ull;
    if (c0 + lane < n) {
      const uint64_t e = region[c0 + lane];
      k = make_key(__uint_as_float((uint32_t)e), (uint32_t)(e >> 32));
    }
    const uint64_t srt = sel::wave_sort64(k, fresh);
    list = fresh ? srt : sel::merge_halves(list, srt, true, tail, c);
    fresh = false;
  }
}

__device__ inline uint64_t readlane64(uint64_t v, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, l);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

// a value slightly below v (v finite): comparing x > below(v) keeps x == v
__device__ inline float below(float v) { return v - (fabsf(v) * 0x1p-20f + 0x1p-126f); }

template <typename T, typename TWP = void>
__global__ __launch_bounds__(kScanThreads) void scan_wave_kernel(
    const T *__restrict__ logits, ScanGeom g, float c, uint64_t *__restrict__ ckeys,
    float2 *__restrict__ ctail, int32_t *__restrict__ cflag, int32_t *__restrict__ zero_ptr,
    int zero_n, HeadProj hp) {
  constexpr int EPL = Elem<T>::EPL;
  constexpr int NL = Raw<T>::NL;
  constexpr int STEP = kScanThreads * EPL;
  constexpr float NINF = -__builtin_huge_valf();
  constexpr int kBufs = WaveScan<T>::kBufs;
  constexpr int kWaveRegion = WaveScan<T>::kRegion;
  __shared__ alignas(16) uint64_t regions[kWaves * kWaveRegion];
  __shared__ uint64_t wl[kWaves][64];
  __shared__ float wthr[kWaves];
  __shared__ float2 red[kWaves];
  __shared__ int flag;
  static_assert(kWaves * kWaveRegion * 8 >= kWaves * 256 * 4, "projection partials fit the regions");
  if constexpr (!std::is_void<TWP>::value) {
    if ((int)blockIdx.x >= g.nchunks) {
      head_proj_tile<TWP>(hp, g.rows, blockIdx.y * hp.extra + blockIdx.x - g.nchunks,
                          reinterpret_cast<float *>(regions));
      return;
    }
  }
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int row = blockIdx.y, seg = blockIdx.x;
  const int M = g.M;
  const int seg_start = seg * g.chunk;
  const int seg_n = min(g.chunk, g.V - seg_start);
  const int nbat = (seg_n + kScanChunk - 1) / kScanChunk;
  const T *rowp = logits + (size_t)row * g.V + seg_start;
  if (zero_ptr && blockIdx.x == 0 && blockIdx.y == 0)
    for (int i = tid; i < zero_n; i += kScanThreads) zero_ptr[i] = 0;
  const __amdgpu_buffer_rsrc_t segr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<T *>(rowp), 0, seg_n * (int)sizeof(T), 0x00020000);
  // loads past the segment's end return zeros (no traffic); pad_batch makes them -inf
  int lb = tid * EPL;
  asm volatile("" : "+v"(lb));
  Raw<T> ra, rb, rc;
  const bool two = nbat > 1;
  load_batch_vec<T>(ra, segr, 0);
  if (two) load_batch_vec<T>(rb, segr, 1);
  if (tid == 0) flag = 0;

  // ---- the first two batches' lower bound tb (every wave: the ceil(M/4)-th
  // largest of its lane maxima; the minimum over the waves).
  // (Two batches rather than one: the bound then admits about 40% fewer
  // candidates over a segment of eight batches, and every candidate costs an
  // append and a share of a merge.)
  const int bn0 = min(kScanChunk, seg_n);
  if (bn0 < kScanChunk) pad_batch<T>(ra, bn0);
  float tmax = NINF;
#pragma unroll
  for (int j = 0; j < NL; ++j)
#pragma unroll
    for (int e = 0; e < EPL; ++e) tmax = fmaxf(tmax, elem<T>(ra, j, e));
  if (two) {
    const int bn1 = min(kScanChunk, seg_n - kScanChunk);
    if (bn1 < kScanChunk) pad_batch<T>(rb, bn1);
#pragma unroll
    for (int j = 0; j < NL; ++j)
#pragma unroll
      for (int e = 0; e < EPL; ++e) tmax = fmaxf(tmax, elem<T>(rb, j, e));
  }
  {
    const int q = (M + kWaves - 1) / kWaves;
    const uint32_t code = ordered_bits(tmax);
    uint32_t pre = 0;
#pragma unroll
    for (int bit = 31; bit >= kLowBit<T>; --bit) {
      const uint32_t cand = pre | (1u << bit);
      if (__popcll(__ballot(code >= cand)) >= q) pre = cand;
    }
    pre = full_code<T>(pre);
    if (lane == 0) wthr[w] = ordered_to_float(pre);
  }
  __syncthreads();
  // the batch after them (issued after the barrier, which would wait for it)
  if constexpr (kBufs == 3) load_batch_vec<T>(rc, segr, 2);
  float tb = wthr[0];
#pragma unroll
  for (int i = 1; i < kWaves; ++i) tb = fminf(tb, wthr[i]);
  const bool all_in = !(tb > NINF);
  const float tlow = all_in ? NINF : below(tb);
  // The tail's reference follows the bound, which every element the tail
  // takes lies at or below, not the segment's maximum: at a small
  // temperature (c large) the tail's terms against the maximum of the
  // candidates would all underflow.
  Tail tail = sel::tail_empty();
  tail.m = fmaxf(tlow, -3.402823466e38f);

  uint64_t list = 0ull;   // this wave's best keys (0: empty)
  bool fresh = true;      // no merge yet (the list is empty)
  float v_own = NINF;     // its M-th value once it holds M keys
  int wpos = 0;           // candidates in the region (wave-uniform)
  const int kMergeTrig = M < 16 ? 2 * M : 48;
  uint64_t *region = regions + w * kWaveRegion;

  auto after_merge = [&]() {
    const uint64_t km = readlane64(list, M - 1);
    if (km) v_own = key_value(km);
  };
  auto merge_now = [&]() {
    wave_merge(region, wpos, list, fresh, tail, c);
    wpos = 0;
    after_merge();
  };
  // the candidates of batch b read again from memory, merged whenever the
  // region might overflow (the tail already holds the batch's other elements)
  auto slow = [&](int bstart, int bn, float te, bool in_all) {
#pragma unroll 1
    for (int k = 0; k < NL * EPL; ++k) {
      const int off = lb + (k / EPL) * STEP + k % EPL;
      const float x = off < bn ? to_f32<T>(rowp[bstart + off]) : NINF;
      const bool pass = off < bn && (x > te || (in_all && x == NINF));
      if (in_all && off < bn && x != x) tail.s = x;  // (a NaN: the row is flagged)
      const uint64_t bal = __ballot(pass);
      if (bal) {
        if (wpos + 64 > kWaveRegion) merge_now();
        const int at = wpos + __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                        __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0));
        if (pass)
          region[at] = ((uint64_t)(uint32_t)(seg_start + bstart + off) << 32) | __float_as_uint(x);
        wpos += __popcll(bal);
      }
    }
  };

  auto process = [&](Raw<T> &raw, int b) {
    const int bstart = b * kScanChunk;
    const int bn = min(kScanChunk, seg_n - bstart);
    if (b > 0 && bn < kScanChunk) pad_batch<T>(raw, bn);
    // this batch's bound
    float te = tlow;
    if (b > 0) te = fmaxf(te, v_own);
    // every element that cannot enter is <= te: keep the tail's reference above it
    if (te > tail.m) {
      tail.s *= sel::fast_exp2((tail.m - te) * c);
      tail.m = te;
    }
    if (b == 0 && all_in) {
      slow(bstart, bn, NINF, true);
    } else {
      fence_regs<T>(raw);
      const int wprev = wpos;
      const int ibase = seg_start + bstart + lb;  // row index of this thread's element (0, 0)
      // exp((x - m) / tau) = 2^((x - m) c) for every element; a candidate (x >
      // te, rare) is appended to the region and adds nothing
      auto tail_pass = [&](auto expo) {
        float s = 0.0f;
#pragma unroll
        for (int j = 0; j < NL; ++j)
#pragma unroll
          for (int e = 0; e < EPL; ++e) {
            float x = elem<T>(raw, j, e);
            const bool pass = x > te;
            const uint64_t bal = __ballot(pass);
            if (__builtin_expect(bal != 0, 0)) {
              // (past the region's end the last slot is overwritten: the
              // overflow below discards this batch's entries)
              const int at = min(wpos + (int)__builtin_amdgcn_mbcnt_hi(
                                            (uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0)),
                                 kWaveRegion - 1);
              if (pass)
                region[at] = ((uint64_t)(uint32_t)(ibase + j * STEP + e) << 32) | __float_as_uint(x);
              wpos += __popcll(bal);
              x = pass ? NINF : x;
            }
            s += sel::fast_exp2(expo(x));
            // (group by group: the sum pinned here keeps the scheduler from
            // holding every converted element at once)
            if (e == EPL - 1) asm volatile("" : "+v"(s));
          }
        tail.s += s;
      };
      const float m = tail.m, mc = m * c;
      if (fabsf(mc) <= 128.0f)
        tail_pass([=](float x) { return __builtin_fmaf(x, c, -mc); });
      else
        tail_pass([=](float x) { return (x - m) * c; });
      if (wpos > kWaveRegion) {
        // overflow: merge what came before, then this batch's candidates again
        wpos = wprev;
        if (wpos) merge_now();
        slow(bstart, bn, te, false);
      }
    }
    if (wpos >= kMergeTrig || (wpos && b == nbat - 1)) merge_now();
  };

  // a buffer is refilled with the batch kBufs ahead as soon as it is processed
  // (loads past the segment's end return zeros and cost no traffic)
  for (int b = 0; b < nbat; b += kBufs) {
    process(ra, b);
    if (b + kBufs < nbat) load_batch_vec<T>(ra, segr, b + kBufs);
    if (b + 1 < nbat) {
      process(rb, b + 1);
      if (b + 1 + kBufs < nbat) load_batch_vec<T>(rb, segr, b + 1 + kBufs);
    }
    if constexpr (kBufs == 3) {
      if (b + 2 < nbat) {
        process(rc, b + 2);
        if (b + 2 + kBufs < nbat) load_batch_vec<T>(rc, segr, b + 2 + kBufs);
      }
    }
  }

  // ---- the four wave lists meet: the segment's M best, the rest to the tail
  // (waves 0 and 2 merge the pairs side by side, wave 2's result ascending;
  // wave 0 merges the two)
  wl[w][lane] = list;
  __syncthreads();
  const size_t cidx = (size_t)row * g.nchunks + seg;
  if ((w & 1) == 0) wl[w][lane] = sel::merge_halves(wl[w][lane], wl[w + 1][63 - lane], w == 0, tail, c);
  __syncthreads();
  if (w == 0) {
    uint64_t f = sel::merge_halves(wl[0][lane], wl[2][lane], true, tail, c);
    if (lane >= M) {
      if (f) sel::tail_add1(tail, key_value(f), c);
      f = 0ull;
    }
    if (lane < M) ckeys[cidx * M + lane] = f;
    // +inf heads the list
    if (lane == 0 && f && key_value(f) == __builtin_huge_valf()) atomicOr(&flag, 1);
  }
  // a NaN makes a tail sum NaN (it never passes a comparison)
  if (!(tail.s == tail.s)) atomicOr(&flag, 1);
  const Tail t = sel::block_tail<kScanThreads>(tail, c, red);
  if (tid == 0) {
    ctail[cidx] = make_float2(t.m, t.s);
    cflag[cidx] = flag ? DT_TREE_NONFINITE : 0;
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
  // segments of sb batches: the fewest rounds of kScanSlots resident
  // workgroups (each round pays a workgroup's start-up latency once; within a
  // round the scan streams at the memory's rate whatever the split), then the
  // shortest segments that keep it (the most workgroups in flight)
  const int nb = (V + kScanChunk - 1) / kScanChunk;
  auto rounds = [&](int t) { return ((long long)rows * ((nb + t - 1) / t) + kScanSlots - 1) / kScanSlots; };
  const long long fewest = rounds(nb);
  int sb = 1;
  while (sb < nb && rounds(sb) > fewest) ++sb;
  g.chunk = sb * kScanChunk;
  g.nchunks = (V + g.chunk - 1) / g.chunk;
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

// hipLaunchKernelGGL, or hipExtLaunchKernelGGL with start and end events
template <typename F, typename... Args>
static void launch_maybe_timed(F kernel, dim3 grid, dim3 block, uint32_t lds, hipStream_t s,
                               hipEvent_t t0, hipEvent_t t1, Args... args) {
  if (t0)
    hipExtLaunchKernelGGL(kernel, grid, block, lds, s, t0, t1, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, lds, s, args...);
}

template <typename T, bool VEC>
static void launch_scan_t(const T *p, const ScanGeom &g, float c, const Workspace &ws, int32_t *zero_ptr,
                          int zero_n, const HeadProj *hp, hipStream_t s, hipEvent_t t0, hipEvent_t t1) {
  const dim3 block(kScanThreads);
  if (VEC && g.M <= 64) {
    // the wave-streaming kernel
    if (!hp) {
      launch_maybe_timed(scan_wave_kernel<T>, dim3(g.nchunks, g.rows), block, 0, s, t0, t1, p, g, c,
                         ws.chunk_keys, ws.chunk_tail, ws.chunk_flag, zero_ptr, zero_n, HeadProj{});
      return;
    }
    const dim3 grid(g.nchunks + hp->extra, g.rows);
    if (hp->wdt == DT_BF16)
      launch_maybe_timed(scan_wave_kernel<T, uint16_t>, grid, block, 0, s, t0, t1, p, g, c, ws.chunk_keys,
                         ws.chunk_tail, ws.chunk_flag, zero_ptr, zero_n, *hp);
    else
      launch_maybe_timed(scan_wave_kernel<T, float>, grid, block, 0, s, t0, t1, p, g, c, ws.chunk_keys,
                         ws.chunk_tail, ws.chunk_flag, zero_ptr, zero_n, *hp);
    return;
  }
  if (!hp) {
    launch_maybe_timed(scan_chunk_kernel<T, VEC>, dim3(g.nchunks, g.rows), block, 0, s, t0, t1, p, g, c,
                       ws.chunk_keys, ws.chunk_tail, ws.chunk_flag, zero_ptr, zero_n, HeadProj{});
    return;
  }
  const dim3 grid(g.nchunks + hp->extra, g.rows);
  if (hp->wdt == DT_BF16)
    launch_maybe_timed(scan_chunk_kernel<T, VEC, uint16_t>, grid, block, 0, s, t0, t1, p, g, c, ws.chunk_keys,
                       ws.chunk_tail, ws.chunk_flag, zero_ptr, zero_n, *hp);
  else
    launch_maybe_timed(scan_chunk_kernel<T, VEC, float>, grid, block, 0, s, t0, t1, p, g, c, ws.chunk_keys,
                       ws.chunk_tail, ws.chunk_flag, zero_ptr, zero_n, *hp);
}

HeadProj head_proj_args(const dt_plan *p, int rows, const void *H, const dt_domino_head &hd, float *a_out) {
  HeadProj h;
  h.w1 = hd.w1;
  h.H = H;
  h.a = a_out;
  h.d_H = hd.d_H;
  h.ld1 = hd.d_H + p->d_h;
  h.rank = hd.rank;
  h.wdt = p->wdt;
  const int tiles = ((hd.rank + 15) / 16) * ((rows + 15) / 16);
  h.extra = (tiles + rows - 1) / rows;
  return h;
}

hipError_t launch_scan_chunks(const void *logits, int ldt, const ScanGeom &g, float inv_tau,
                              const Workspace &ws, int32_t *zero_ptr, int zero_n, hipStream_t s,
                              hipEvent_t t0, hipEvent_t t1, const HeadProj *hp) {
  const float c = 1.4426950408889634f * inv_tau;  // exp(x / tau) = exp2(x * c)
  const bool aligned = (reinterpret_cast<uintptr_t>(logits) % 16) == 0;
  if (ldt == DT_BF16) {
    const uint16_t *p = static_cast<const uint16_t *>(logits);
    if (aligned && g.V % 8 == 0)
      launch_scan_t<uint16_t, true>(p, g, c, ws, zero_ptr, zero_n, hp, s, t0, t1);
    else
      launch_scan_t<uint16_t, false>(p, g, c, ws, zero_ptr, zero_n, hp, s, t0, t1);
  } else {
    const float *p = static_cast<const float *>(logits);
    if (aligned && g.V % 4 == 0)
      launch_scan_t<float, true>(p, g, c, ws, zero_ptr, zero_n, hp, s, t0, t1);
    else
      launch_scan_t<float, false>(p, g, c, ws, zero_ptr, zero_n, hp, s, t0, t1);
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
