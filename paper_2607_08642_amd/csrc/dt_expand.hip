// S3-S5: best-first conditional expansion and emission (Alg. 1 steps 2-4;
// section 3.1 conditional children; section 3.5 verification mask), preceded
// by the per-row merge of the scan (Alg. 1 step 1).
//
// The heap of Alg. 1 pops nodes in non-increasing score order, and a child
// never scores above its parent (log-probs are <= 0), so the popped set is the
// top-B of the candidate tree (the frontier argument of Appendix B).  A node
// scoring below the B-th best score already known can never be popped.  The
// kernel uses this in two phases:
//
//  A. Speculative, depth-synchronous expansion.  Starting from the root,
//     every known node that is not expanded, is above depth L and scores at
//     least the current B-th best known score is expanded, up to 16 nodes at a
//     time: the GRU advances its path state (split-bf16 MFMA against W_hh,
//     fp32 accumulation; fp32 MFMA for fp32 weights), the correction of the next
//     depth's slice is an fp32 MFMA against the gathered rows U[v] = W_c^T E[v],
//     and the top-k children are appended.  This repeats until no node
//     qualifies; every node the heap can pop below depth L is then expanded.
//  B. Exact replay of the heap: B pops by (score desc, insertion order asc),
//     where insertion order is (parent's pop index, child rank) -- the order in
//     which Alg. 1 pushes.  Ties therefore resolve exactly as in the heap.
//
// A tree is built by a group of G workgroups.  Member j owns hidden units
// [j*d_h/G, (j+1)*d_h/G): it advances those units of every path state and
// forms the part of each correction dot product that runs over them.  The
// parts meet through global memory with device-scope (sc1) stores and
// vectorised device-scope buffer loads, after a relaxed-atomic counter barrier
// per expansion step; every member then
// sums the parts in the same order and runs the same bookkeeping, so all
// members hold identical node tables without further exchange.  The members
// of a group are placed on one XCD (blocks are dealt to XCDs round-robin).
// Member 0 replays the heap and emits the tree.
#include "dt_select.h"
#include <hip/hip_ext.h>

#include <type_traits>

namespace dt {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int NT = kExpThreads;
constexpr int NW = NT / 64;
constexpr int NC = kNodeCap;
constexpr int CH = kChunkNodes;
constexpr int kSpinLimit = 1 << 18;  // default bound of a wait (~0.3 s): longer means a fault
static_assert(CH == 16, "MFMA column count");
static_assert(CH == 2 * NW, "children step: two nodes per wave");

struct ExpArgs {
  int L, M, B, k, dh, G, norm_mode, pos_offset, ecap, batch, nchunks, nxcd;
  int W;           // frontier width (Appendix B's frontier builder); 0: the heap of Alg. 1
  int use_ids;     // every row's candidate ids staged in LDS (the U slices, or Domino's head)
  // Domino's own head (section 2.3; HEAD instances): delta_m = W_2[cand_m] . y,
  // y = SiLU(a_d + W_1^S S); member j owns the rank slice [j RJ, (j + 1) RJ)
  int rank, RJ, ld1, d_H;
  const void *w1;   // [rank][ld1] (weights dtype); columns d_H .. d_H + dh act on S
  const void *w2;   // [V][rank] (weights dtype)
  const float *ha;  // [batch * L][rank] a_d = W_1^H H_d
  float *hpart;     // [batch][2][G][CH][rank] partial W_1^S S of each member
  int spin_limit;  // polls before a cross-workgroup wait gives up (DT_TREE_TIMEOUT)
  int use_us;  // U slices of the expanded depth staged into LDS (see us_fits)
  // ablation-arm modes (ExpMode): no correction (the marginals, or menu_in's
  // per-depth menus); menu_out: every expanded node's slot log-probs; emit = 0:
  // no replay or emission; skip_merge: the rows are already merged
  int nocorr, emit, skip_merge;
  const float *menu_in;  // [batch][L][MP]
  float *menu_out;       // [batch][L][MP]
  int32_t *stats;        // [batch][2] expansion steps and expanded nodes per tree, or null
  const float *cost;     // adaptive budget: C_d, C_v(0..B) (device), or null (fixed budget)
  float inv_tau, c2;  // c2 = log2(e) / tau
  const uint64_t *ckeys;
  const float2 *ctail;
  const int32_t *cflag;
  int32_t *cand;   // [rows][M] merged rows (written by the group, read by all members)
  float *candv;    // [rows][M]
  float *tailR;    // [rows]
  int32_t *rflag;  // [rows]
  const float *P_all;  // [V][3dh] W_ih E[v] + b_ih
  const float *U_all;  // [V][dh]  W_c^T E[v]
  const float *c_all;  // [V]      E[v] . b_c
  const void *whh;
  const float *b_hh;
  const float *h0;
  float *states;   // [batch][ecap][dh] path states of expanded nodes; slot ecap-1: the root
  float *part;     // [batch][2][G][CH][MP] partial corrections
  int32_t *bar;    // [batch + kSlotRows][kBarStride] barrier and slot counters (zeroed by the scan kernel)
  dt_tree out;
};

// LDS carve (byte offsets), identical on host and device
// Scores kept beside the candidate lists (elist, elist2): the list's first
// kCsCap entries.  After an expansion step the list holds the old candidates
// and then the step's new children, whose scores are ranked in place.
constexpr int kCsCap = 512;

struct Lds {
  int ng, ntok, nparent, nstate, nslot, ndepth, nrank, nexp, newidx, elist, elist2, cs, cs2;
  int ins, popd, ppi, order, anc;
  int rcand, rcandv;  // the merged row of the depth being expanded
  int rowids, uslice;  // all rows' candidate ids; this member's U slice of one depth
  int pin, bhn;        // GRU inputs P of the chunk's nodes (this member's units); b_hn
  int hw2, hys, ha;    // Domino's head: W_2 rows (rank slice, weights dtype), y slice, a_d slice
  int gpart, Sp, Sn, ell, rnk, chunk, scal, total;
  int sortbuf;  // aliases gpart.. (prologue only)
};

__host__ __device__ inline int mp_of(int M) { return (M + 63) / 64 * 64; }
// Row stride (floats) of the parent states staged in LDS: rows of d_h = 256 n
// floats would put a lane group's 16 nodes on one bank (the MFMA B operand
// reads one row per lane); four floats of padding spread them over all banks.
// (The staging copies 256 floats per instruction, so only then can a row be
// padded.)
__host__ __device__ inline int sp_stride(int dh) { return dh % 256 == 0 ? dh + 4 : dh; }

// The U rows of a depth's candidates (this member's units) are staged into LDS
// with the parent states when the slice and all rows' ids are small.
// The GRU inputs (rows of P, gates r, z, n) of a chunk's nodes are staged into
// LDS when this member's slice is small; W_hh fragments are then loaded ahead.
// Each node's three UW-float rows take one 256-float slot (one wave instruction).
constexpr int kPinSlot = 256;
__host__ __device__ inline bool pin_fits(int dh, int G) { return 3 * (dh / G) <= kPinSlot; }
__host__ __device__ inline bool us_fits(int dh, int G, int M, int L) {
  const int MP = mp_of(M);
  return MP * (dh / G) * 4 <= 16384 && L * MP * 4 <= 8192;
}

// rj > 0: a HEAD instance with rank slice rj and weights of wbytes bytes
__host__ __device__ inline Lds lds_layout(int dh, int G, int M, int nchunks, int L, int rj = 0,
                                          int wbytes = 0) {
  Lds l;
  int o = 0;
  auto take = [&](int bytes) {
    const int r = o;
    o += (bytes + 15) / 16 * 16;
    return r;
  };
  const int MP = mp_of(M);
  const int UW = dh / G;
  l.ng = take(NC * 4);
  l.ntok = take(NC * 4);
  l.nparent = take(NC * 2);
  l.nstate = take(NC * 2);
  l.nslot = take(NC * 2);
  l.ndepth = take(NC);
  l.nrank = take(NC);
  l.nexp = take(NC);
  l.newidx = take(NC * 2);
  l.elist = take(NC * 2);
  l.elist2 = take(NC * 2);
  l.cs = take(kCsCap * 4);
  l.cs2 = take(kCsCap * 4);
  l.ins = take(NC);
  l.popd = take(NC);
  l.ppi = take(NC * 2);
  l.order = take(kMaxB * 2);
  l.anc = take(kMaxB * 8 * 4);
  l.rcand = take(MP * 4);
  l.rcandv = take(MP * 4);
  const bool us = us_fits(dh, G, M, L);
  l.rowids = take((us || rj) ? L * MP * 4 : 0);
  l.uslice = take(us && !rj ? MP * UW * 4 : 0);
  l.hw2 = take(rj ? MP * rj * wbytes : 0);
  l.hys = take(rj ? CH * rj * 4 : 0);
  l.ha = take(rj ? rj * 4 : 0);
  const bool pin = pin_fits(dh, G);
  l.pin = take(pin ? CH * kPinSlot * 4 : 0);
  l.bhn = take(pin ? UW * 4 : 0);
  l.chunk = take(CH * 2);
  l.scal = take(64 * 4);
  // region reused by the prologue's merge
  const int reuse = o;
  l.gpart = take(UW / 16 < NW ? NW * 3 * 256 * 4 : 0);  // k-split partial gates
  l.Sp = take(CH * sp_stride(dh) * 4);
  l.Sn = take(CH * UW * 4);
  l.ell = take(CH * MP * 4);
  l.rnk = take(CH * MP * 2);
  // merge_row's buffer, or merge_row_tree's (NT keys)
  const int sortb = sel::merge_buf_bytes(nchunks, M) > NT * 8 ? sel::merge_buf_bytes(nchunks, M) : NT * 8;
  l.sortbuf = reuse;
  if (reuse + sortb > o) o = reuse + sortb;
  l.total = o;
  return l;
}

// scalar slots in LDS
enum { S_NN, S_VB, S_NEXP, S_STATUS, S_NCAND, S_NC, S_TOT, S_STOP, S_NPOP, S_R, S_MERGEFLAG, S_SLOT, S_CUR,
       S_NNEXT0, S_NNEXT1 };
// per-wave slots (16-byte aligned: read as two float4)
constexpr int S_CNT0 = 16;
// after the per-wave slots S_CNT0 ..: which candidate buffer holds the list,
// where the last append started, and the list's entries.  The next list's
// count alternates between S_NNEXT0 and S_NNEXT1 from one ranking to the next.
static_assert(kExpThreads / 64 == 8, "eight per-wave slots");
constexpr int S_CLIST = S_CNT0 + kExpThreads / 64;
constexpr int S_ABASE = S_CLIST + 1;
constexpr int S_NVAL = S_CLIST + 2;  // entries of the current list: candidates, then new children
static_assert(S_NVAL + 1 <= 32, "scalar slots below the reduction area");


// GRU activations on the hardware exp2 and reciprocal (about 1 ulp each):
// sigmoid(x) = 1 / (1 + 2^(-x log2 e)), tanh(x) = 2 sigmoid(2x) - 1 (absolute
// error ~1e-7, far below the path-state tolerance)
__device__ inline float sigmoid_fast(float x) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.44269504088896341f * x));
}
__device__ inline float tanh_fast(float x) { return 2.0f * sigmoid_fast(2.0f * x) - 1.0f; }
// e^x and ln x on the hardware exp2 / log2 (about 1 ulp; x <= 0 and x >= 1 here)
__device__ inline float exp_hw(float x) { return __builtin_amdgcn_exp2f(1.44269504088896341f * x); }
__device__ inline float log_hw(float x) { return 0.69314718055994531f * __builtin_amdgcn_logf(x); }

__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

template <typename T>
__device__ inline T ld_dev(const T *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ inline void st_dev(T *p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Device-scope (sc1) vector loads of data other workgroups wrote.  Plain
// (non-atomic) buffer loads, so the compiler batches them; `base` must be
// uniform across the wave, the byte offset may vary per lane.
__device__ inline __amdgpu_buffer_rsrc_t dev_rsrc(const void *base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, 0x7FFFFFF0, 0x00020000);
}
constexpr int kSc1 = 16;  // cache-policy bit: device scope
__device__ inline float4 ld_dev16(__amdgpu_buffer_rsrc_t r, int byte_off, int sgpr_off = 0) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, sgpr_off, kSc1));
}
__device__ inline float ld_dev4(__amdgpu_buffer_rsrc_t r, int byte_off, int sgpr_off = 0) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, byte_off, sgpr_off, kSc1));
}
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Partial corrections of 64 slots from up to 16 members, four 16-byte loads
// per lane: lane (q = lane % 16, r = lane / 16) holds slots 4q .. 4q+3 of
// members r, r+4, r+8, r+12 (zeros for members >= G).
struct Parts {
  float4 v[4];
};
__device__ inline float lane_pull(float v, int src_lane) {
  return __builtin_bit_cast(float,
                            __builtin_amdgcn_ds_bpermute(src_lane * 4, __builtin_bit_cast(int, v)));
}
// The sum of the G parts of slot `lane`, bit-identical in every member: each
// lane adds its members in the order r, r+4, r+8, r+12; lane groups {r, r^2}
// then {r, r^1} combine (each slot's sum is formed in one lane, slot 4q + r
// in lane (q, r)), and lane l finally takes slot l.
__device__ inline float sum_parts(const Parts &p, int lane) {
  const float4 t = ((p.v[0] + p.v[1]) + p.v[2]) + p.v[3];
  const bool hi = lane >= 32, odd = (lane >> 4) & 1;
  // r, r^2: the low pair keeps slots 4q, 4q+1, the high pair 4q+2, 4q+3
  const float h0 = (hi ? t.z : t.x) + lane_pull(hi ? t.x : t.z, lane ^ 32);
  const float h1 = (hi ? t.w : t.y) + lane_pull(hi ? t.y : t.w, lane ^ 32);
  // r, r^1: lane r keeps slot 4q + r
  const float tot = (odd ? h1 : h0) + lane_pull(odd ? h0 : h1, lane ^ 16);
  return lane_pull(tot, (lane >> 2) + 16 * (lane & 3));
}

// GRU inputs of 4 consecutive hidden units j0..j0+3 of one node: P of gates
// r, z, n (P = the token's folded input projection) and b_hn
struct GruIn {
  float4 r, z, n, b;
};
__device__ inline GruIn load_gru_in(const float *prow, const float *b_hh, int dh, int j0) {
  GruIn g;
  g.r = *reinterpret_cast<const float4 *>(prow + j0);
  g.z = *reinterpret_cast<const float4 *>(prow + dh + j0);
  g.n = *reinterpret_cast<const float4 *>(prow + 2 * dh + j0);
  g.b = *reinterpret_cast<const float4 *>(b_hh + 2 * dh + j0);
  return g;
}
// four consecutive weights as stored (bf16: 8 bytes; fp32: 16 bytes), and widened
template <typename TW>
struct W4;
template <>
struct W4<uint16_t> {
  using T = uint2;
  static __device__ inline T load(const uint16_t *p) { return *reinterpret_cast<const uint2 *>(p); }
  static __device__ inline float4 widen(T q) {
    return make_float4(__uint_as_float(q.x << 16), __uint_as_float(q.x & 0xFFFF0000u),
                       __uint_as_float(q.y << 16), __uint_as_float(q.y & 0xFFFF0000u));
  }
};
template <>
struct W4<float> {
  using T = float4;
  static __device__ inline T load(const float *p) { return *reinterpret_cast<const float4 *>(p); }
  static __device__ inline float4 widen(T q) { return q; }
};
// four consecutive weights widened to fp32 (bf16: 8 bytes; fp32: 16 bytes)
__device__ inline float4 load4w(const uint16_t *p) {
  const uint2 q = *reinterpret_cast<const uint2 *>(p);
  return make_float4(__uint_as_float(q.x << 16), __uint_as_float(q.x & 0xFFFF0000u),
                     __uint_as_float(q.y << 16), __uint_as_float(q.y & 0xFFFF0000u));
}
__device__ inline float4 load4w(const float *p) { return *reinterpret_cast<const float4 *>(p); }
__device__ inline void st_dev16(__amdgpu_buffer_rsrc_t r, int byte_off, float4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, byte_off, 0, kSc1);
}

__device__ inline uint64_t wave_max_u64(uint64_t v) {
  auto mx = [](uint64_t x, uint64_t y) { return x > y ? x : y; };
  v = mx(v, sel::lane_xor64<32>(v));
  v = mx(v, sel::lane_xor64<16>(v));
  v = mx(v, sel::lane_xor64<8>(v));
  v = mx(v, sel::lane_xor64<4>(v));
  v = mx(v, sel::lane_xor64<2>(v));
  return mx(v, sel::lane_xor64<1>(v));
}
__device__ inline float wave_max_f(float v) {
  return sel::wave_reduce(v, [](float x, float y) { return fmaxf(x, y); });
}
__device__ inline float wave_sum_f(float v) {
  return sel::wave_reduce(v, [](float x, float y) { return x + y; });
}
__device__ inline float wave_min_f(float v) {
  return sel::wave_reduce(v, [](float x, float y) { return fminf(x, y); });
}

// inclusive prefix sum over each row of 16 lanes (DPP row shifts; a lane
// whose source lies outside the row adds 0)
__device__ inline int row_prefix16(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, false);  // row_shr:8
  return x;
}

// ordered exclusive prefix of a predicate over the block (wcnt: NW ints in LDS)
struct Compact {
  int pos;
  int total;
};
__device__ inline Compact block_compact(bool pred, int *wcnt) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const uint64_t b = __ballot(pred);
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  if (lane == 0) wcnt[w] = __popcll(b);
  __syncthreads();
  int base = 0, tot = 0;
  for (int i = 0; i < NW; ++i) {
    const int c = wcnt[i];
    if (i < w) base += c;
    tot += c;
  }
  __syncthreads();
  return Compact{base + (int)__popcll(b & below), tot};
}

// Relaxed-atomic barrier of the G members of a tree.  Each thread first waits
// for its own stores (device-scope stores are then visible at device scope).
__device__ inline void group_barrier(int32_t *ctr, int G, int &nbar, int *status, int limit) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  ++nbar;
  if (G > 1 && threadIdx.x == 0) {
    __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int target = G * nbar;
    int spins = 0;
    while (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      if (++spins > limit) {
        *status |= DT_TREE_TIMEOUT;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  __syncthreads();
}

// W_hh . S for one group of 16 hidden units (gates r, z, n) over ks in [ks0, ks1).
// B operand: lane l holds S[node l%16][32 ks + 8 (l/16) + e] from the LDS
// staging of the parent states (row stride dh).
template <typename TW>
struct Gates;

template <>
struct Gates<uint16_t> {  // bf16 W_hh: 16x16x32 bf16 MFMA, S split as hi + mid + lo
  // a k range of up to kPre steps can have its weights loaded ahead of time
  static constexpr int kPre = 4;
  struct Pre {
    uint4 w[kPre][3];
  };
  static __device__ inline void preload(const ExpArgs &a, int u, int ks0, int ks1, Pre &p) {
    const int lane = threadIdx.x & 63;
    const int nks = a.dh / 32;
    const uint4 *W = static_cast<const uint4 *>(a.whh);
#pragma unroll
    for (int kk = 0; kk < kPre; ++kk)
#pragma unroll
      for (int g = 0; g < 3; ++g)
        if (ks0 + kk < ks1) p.w[kk][g] = W[((size_t)(u * 3 + g) * nks + ks0 + kk) * 64 + lane];
  }
  static __device__ inline void step(const float *srow, int ks, const uint4 (&wv)[3],
                                     f32x4 (&acc)[3]) {
    const float4 s0 = *reinterpret_cast<const float4 *>(srow + ks * 32);
    const float4 s1 = *reinterpret_cast<const float4 *>(srow + ks * 32 + 4);
    const float x[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
    // S = hi + mid + lo, each rounded to nearest (v_cvt_pk_bf16_f32); the
    // residuals are exact, so the three bf16 products carry S to fp32 accuracy
    bf16x8 hi, mi, lo;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const __bf16 h = (__bf16)x[e];
      const float r1 = x[e] - (float)h;
      const __bf16 m = (__bf16)r1;
      hi[e] = h;
      mi[e] = m;
      lo[e] = (__bf16)(r1 - (float)m);
    }
#pragma unroll
    for (int g = 0; g < 3; ++g) {
      const bf16x8 wa = __builtin_bit_cast(bf16x8, wv[g]);
      acc[g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, lo, acc[g], 0, 0, 0);
      acc[g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, mi, acc[g], 0, 0, 0);
      acc[g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, hi, acc[g], 0, 0, 0);
    }
  }
  // k steps [ks0, ks1) from preload(a, u, ks0, ks1, p); ks1 - ks0 <= kPre
  static __device__ inline void run_pre(const ExpArgs &a, const float *Sp, const Pre &p, int ks0,
                                        int ks1, f32x4 (&acc)[3]) {
    const int lane = threadIdx.x & 63;
    const float *srow = Sp + (lane & 15) * sp_stride(a.dh) + (lane >> 4) * 8;
#pragma unroll
    for (int g = 0; g < 3; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < kPre; ++kk)
      if (ks0 + kk < ks1) step(srow, ks0 + kk, p.w[kk], acc);
  }
  static __device__ inline void run(const ExpArgs &a, const float *Sp, int u, int ks0, int ks1,
                                    f32x4 (&acc)[3]) {
    const int lane = threadIdx.x & 63;
    const int nks = a.dh / 32;
    const uint4 *W = static_cast<const uint4 *>(a.whh);
    const float *srow = Sp + (lane & 15) * sp_stride(a.dh) + (lane >> 4) * 8;
#pragma unroll
    for (int g = 0; g < 3; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
    constexpr int PF = 2;  // k-steps of weights in flight at once
    for (int k0 = ks0; k0 < ks1; k0 += PF) {
      uint4 wv[PF][3];
#pragma unroll
      for (int kk = 0; kk < PF; ++kk)
#pragma unroll
        for (int g = 0; g < 3; ++g)
          if (k0 + kk < ks1) wv[kk][g] = W[((size_t)(u * 3 + g) * nks + k0 + kk) * 64 + lane];
#pragma unroll
      for (int kk = 0; kk < PF; ++kk) {
        if (k0 + kk >= ks1) break;
        step(srow, k0 + kk, wv[kk], acc);
      }
    }
  }
};

template <>
struct Gates<float> {  // fp32 W_hh: 16x16x4 fp32 MFMA, k-groups of 16, two per ks
  static constexpr int kPre = 0;  // no weights loaded ahead (too many registers)
  struct Pre {};
  static __device__ inline void preload(const ExpArgs &, int, int, int, Pre &) {}
  static __device__ inline void run_pre(const ExpArgs &, const float *, const Pre &, int, int,
                                        f32x4 (&acc)[3]) {
#pragma unroll
    for (int g = 0; g < 3; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};  // never called
  }
  static __device__ inline void run(const ExpArgs &a, const float *Sp, int u, int ks0, int ks1,
                                    f32x4 (&acc)[3]) {
    const int lane = threadIdx.x & 63;
    const int nq = a.dh / 16;
    const float4 *W = static_cast<const float4 *>(a.whh);
    const float *srow = Sp + (lane & 15) * sp_stride(a.dh) + (lane >> 4) * 4;
#pragma unroll
    for (int g = 0; g < 3; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int q = 2 * ks0; q < 2 * ks1; ++q) {
      const float4 x = *reinterpret_cast<const float4 *>(srow + q * 16);
#pragma unroll
      for (int g = 0; g < 3; ++g) {
        const float4 wv = W[((size_t)(u * 3 + g) * nq + q) * 64 + lane];
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(wv.x, x.x, acc[g], 0, 0, 0);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(wv.y, x.y, acc[g], 0, 0, 0);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(wv.z, x.z, acc[g], 0, 0, 0);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(wv.w, x.w, acc[g], 0, 0, 0);
      }
    }
  }
};

// SDH, SG, SM, SL > 0 fix d_h, G, M and L at compile time (the LDS layout and
// every loop bound over them become constants); 0 takes them from the arguments.
// ARMS compiles the ablation-arm modes in (nocorr, menu_in, menu_out, emit,
// skip_merge); without it they are fixed off and cost nothing.
// HEAD scores with Domino's own head (a different correction; no ablation arms).
template <typename TW, int SDH, int SG, int SM, int SL, bool ARMS, bool HEAD = false>
__global__ __launch_bounds__(NT) void expand_kernel(ExpArgs a) {
  if constexpr (!ARMS) {
    a.nocorr = 0;
    a.emit = 1;
    a.skip_merge = 0;
    a.menu_in = nullptr;
    a.menu_out = nullptr;
  }
  if constexpr (SDH > 0) a.dh = SDH;
  if constexpr (SG > 0) a.G = SG;
  if constexpr (SM > 0) a.M = SM;
  if constexpr (SL > 0) a.L = SL;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const Lds ly = lds_layout(a.dh, a.G, a.M, a.nchunks, a.L, HEAD ? a.RJ : 0, HEAD ? (int)sizeof(TW) : 0);
  float *ng = reinterpret_cast<float *>(smem + ly.ng);
  int32_t *ntok = reinterpret_cast<int32_t *>(smem + ly.ntok);
  int16_t *nparent = reinterpret_cast<int16_t *>(smem + ly.nparent);
  int16_t *nstate = reinterpret_cast<int16_t *>(smem + ly.nstate);
  int16_t *nslot = reinterpret_cast<int16_t *>(smem + ly.nslot);
  uint8_t *ndepth = reinterpret_cast<uint8_t *>(smem + ly.ndepth);
  uint8_t *nrank = reinterpret_cast<uint8_t *>(smem + ly.nrank);
  uint8_t *nexp = reinterpret_cast<uint8_t *>(smem + ly.nexp);
  int16_t *newidx = reinterpret_cast<int16_t *>(smem + ly.newidx);
  int16_t *elist = reinterpret_cast<int16_t *>(smem + ly.elist);
  int16_t *elist2 = reinterpret_cast<int16_t *>(smem + ly.elist2);
  float *cs = reinterpret_cast<float *>(smem + ly.cs);
  float *cs2 = reinterpret_cast<float *>(smem + ly.cs2);
  uint8_t *ins = reinterpret_cast<uint8_t *>(smem + ly.ins);
  uint8_t *popd = reinterpret_cast<uint8_t *>(smem + ly.popd);
  int16_t *ppi = reinterpret_cast<int16_t *>(smem + ly.ppi);
  int16_t *order = reinterpret_cast<int16_t *>(smem + ly.order);
  uint32_t *anc = reinterpret_cast<uint32_t *>(smem + ly.anc);
  float *gpart = reinterpret_cast<float *>(smem + ly.gpart);
  float *Sp = reinterpret_cast<float *>(smem + ly.Sp);
  float *Sn = reinterpret_cast<float *>(smem + ly.Sn);
  float *ell = reinterpret_cast<float *>(smem + ly.ell);
  int16_t *rnk = reinterpret_cast<int16_t *>(smem + ly.rnk);
  int32_t *rcand = reinterpret_cast<int32_t *>(smem + ly.rcand);
  float *rcandv = reinterpret_cast<float *>(smem + ly.rcandv);
  int32_t *rowids = reinterpret_cast<int32_t *>(smem + ly.rowids);
  float *Us = reinterpret_cast<float *>(smem + ly.uslice);
  float *pin = reinterpret_cast<float *>(smem + ly.pin);
  char *hw2 = smem + ly.hw2;
  float *hys = reinterpret_cast<float *>(smem + ly.hys);
  float *has = reinterpret_cast<float *>(smem + ly.ha);
  float *bhn = reinterpret_cast<float *>(smem + ly.bhn);
  int16_t *cl = reinterpret_cast<int16_t *>(smem + ly.chunk);
  int *scal = reinterpret_cast<int *>(smem + ly.scal);
  float *scalf = reinterpret_cast<float *>(smem + ly.scal);
  int *wcnt = scal + 48;
  uint64_t *sortbuf = reinterpret_cast<uint64_t *>(smem + ly.sortbuf);
  float2 *red = reinterpret_cast<float2 *>(scal + 32);
  int *xoff = scal + 32;  // after the prologue: the chunk's nodes' first child offsets

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = a.L, M = a.M, B = a.B, dh = a.dh, G = a.G;
  const int MP = mp_of(M);
  const int UW = dh / G;       // hidden units of this member
  const int NG = UW / 16;      // unit groups of this member
  const int SPS = sp_stride(dh);
  const bool use_pin = pin_fits(dh, G);
  const float NEG_INF = -__builtin_huge_valf();

  // ---- which tree, which member (members of a tree share an XCD) ------------
  // Workgroups take member slots in the order they start running, from one
  // counter per XCD class (blocks are dealt to XCDs round-robin): complete
  // groups form first, so members never wait for a workgroup that cannot be
  // scheduled while the rest of the grid holds the CUs.
  int t, member;
  if (G > 1) {
    const int xcd = blockIdx.x % a.nxcd;
    // (an XCD class without a tree -- tree t lives in class t % nxcd -- leaves
    // at once: its slot could only name a tree >= batch)
    if (xcd >= a.batch) return;
    if (tid == 0)
      scal[S_SLOT] = __hip_atomic_fetch_add(a.bar + a.batch * kBarStride + xcd * kSlotStride, 1,
                                            __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const int kk = scal[S_SLOT];
    t = xcd + a.nxcd * (kk / G);
    member = kk % G;
  } else {
    t = blockIdx.x;
    member = 0;
  }
  if (t >= a.batch) return;
  int32_t *ctr = a.bar + t * kBarStride;
  int nbar = 0;
  const int u0 = member * NG;  // first unit group of this member

  int chunk_cap = (NC - B - 64) / a.k;
  chunk_cap = chunk_cap > CH ? CH : (chunk_cap < 1 ? 1 : chunk_cap);

  if (tid == 0) {
    scal[S_STATUS] = 0;
    scal[S_NN] = 0;
    scalf[S_VB] = NEG_INF;
    scal[S_NEXP] = 0;
    scal[S_STOP] = 0;
    scal[S_CUR] = 0;
    scal[S_NCAND] = 0;  // no candidates yet (vB is -inf)
    scal[S_CLIST] = 0;
    scal[S_ABASE] = 0;
    scal[S_NVAL] = 0;
    scal[S_NNEXT0] = 0;
    scal[S_NNEXT1] = 0;
  }

  __syncthreads();

  // ---- prologue: merge this member's rows of the scan ------------------------
  // (the root's path state, h0 or zeros, is loaded first and stored after)
  static_assert(kMaxDh <= 2 * NT, "root state: two units per thread");
  float h0v[2] = {0.0f, 0.0f};
  const float bhv = (use_pin && tid < UW) ? a.b_hh[2 * dh + member * UW + tid] : 0.0f;  // b_hn
#pragma unroll
  for (int q = 0; q < 2; ++q)
    if (a.h0 && tid + q * NT < UW) h0v[q] = a.h0[(size_t)t * dh + member * UW + tid + q * NT];
  if (a.skip_merge) {
    // (the rows were merged by the call's first expansion launch)
  } else if (sel::wave_merge_fits(a.nchunks, M) && a.nchunks > 2) {
    // all waves on each of this member's rows
    for (int d = member; d < L; d += G) {
      const int row = t * L + d;
      sel::merge_row_tree<true, NT, true>(a.ckeys + (size_t)row * a.nchunks * M, a.nchunks, M,
                                    a.ctail + (size_t)row * a.nchunks, a.cflag + (size_t)row * a.nchunks,
                                    a.c2, a.inv_tau, sortbuf, red, a.cand + (size_t)row * M,
                                    a.candv + (size_t)row * M, a.tailR + row, a.rflag + row, a.c_all);
    }
  } else if (sel::wave_merge_fits(a.nchunks, M)) {
    // one wave per row (a single merge): rows member + G * (wave + NW * i)
    for (int d = member + G * wave; d < L; d += G * NW) {
      const int row = t * L + d;
      sel::merge_row_wave<true, true>(a.ckeys + (size_t)row * a.nchunks * M, a.nchunks, M,
                                a.ctail + (size_t)row * a.nchunks, a.cflag + (size_t)row * a.nchunks,
                                a.c2, a.inv_tau, a.cand + (size_t)row * M, a.candv + (size_t)row * M,
                                a.tailR + row, a.rflag + row, a.c_all);
    }
  } else {
    for (int d = member; d < L; d += G) {
      const int row = t * L + d;
      sel::merge_row<NT, true, true>(a.ckeys + (size_t)row * a.nchunks * M, a.nchunks, M,
                               a.ctail + (size_t)row * a.nchunks, a.cflag + (size_t)row * a.nchunks,
                               a.c2, a.inv_tau, sortbuf, red, &scal[S_MERGEFLAG],
                               a.cand + (size_t)row * M, a.candv + (size_t)row * M, a.tailR + row,
                               a.rflag + row, a.c_all);
    }
  }
  {
    // the root's path state (h0 or zeros) in slot ecap-1: this member's units
    float *root = a.states + ((size_t)t * a.ecap + a.ecap - 1) * dh;
#pragma unroll
    for (int q = 0; q < 2; ++q)
      if (tid + q * NT < UW) st_dev(root + member * UW + tid + q * NT, h0v[q]);
    if (use_pin && tid < UW) bhn[tid] = bhv;
  }
  group_barrier(ctr, G, nbar, &scal[S_STATUS], a.spin_limit);
  // (a wait that gave up: the other members' rows may be missing, so nothing of
  // them is read; the tree is emitted empty below)
  const bool timed_out = scal[S_STATUS] & DT_TREE_TIMEOUT;
  if (!timed_out) {
    // one round trip: the row flags and (U slices staged) every row's candidate ids
    const __amdgpu_buffer_rsrc_t rfl = dev_rsrc(a.rflag + (size_t)t * L);
    const __amdgpu_buffer_rsrc_t rid = dev_rsrc(a.cand + (size_t)t * L * M);
    const int f = tid < L ? __builtin_bit_cast(int, ld_dev4(rfl, tid * 4)) : 0;
    constexpr int kIdsPer = 4;  // L * MP * 4 <= 8192 bytes when U slices are staged
    static_assert(8192 / 4 <= kIdsPer * NT, "row ids per thread");
    int ids[kIdsPer];
#pragma unroll
    for (int q = 0; q < kIdsPer; ++q) {
      const int i = tid + q * NT;
      const int d = i / MP, m = i - d * MP;
      ids[q] = (a.use_ids && i < L * MP && m < M) ? __builtin_bit_cast(int, ld_dev4(rid, (d * M + m) * 4)) : 0;
    }
    if (f) atomicOr(&scal[S_STATUS], f);
#pragma unroll
    for (int q = 0; q < kIdsPer; ++q) {
      const int i = tid + q * NT;
      if (a.use_ids && i < L * MP) rowids[i] = ids[q] > 0 ? ids[q] : 0;  // dead slots (-1) read row 0, unused
    }
  }
  __syncthreads();

  dt_tree o = a.out;
  int32_t *otok = o.tokens + (size_t)t * B;
  int32_t *opar = o.parents + (size_t)t * B;
  int32_t *odep = o.depth + (size_t)t * B;
  int32_t *opos = o.position_ids + (size_t)t * B;
  float *osc = o.scores + (size_t)t * B;
  uint8_t *omask = o.mask + (size_t)t * B * B;

  // a tree with no nodes: non-finite logits, or a wait that gave up
  auto emit_empty = [&]() {
    for (int i = tid; i < B; i += NT) {
      otok[i] = -1;
      opar[i] = -1;
      odep[i] = 0;
      opos[i] = a.pos_offset;
      osc[i] = NEG_INF;
    }
    for (int i = tid; i < B * B; i += NT) omask[i] = 0;
    if (tid == 0) {
      o.n_nodes[t] = 0;
      o.status[t] = scal[S_STATUS];
    }
  };
  if (scal[S_STATUS] & (DT_TREE_NONFINITE | DT_TREE_TIMEOUT)) {
    if (member == 0 && a.emit) emit_empty();
    return;
  }

  // ---- one expansion step: up to 16 nodes, all at depth d (d = 0: the root) ---
  // this wave's share of W_hh . S: unit group gu (-1: none) over k steps [gk0, gk1);
  // when that fits kPre k steps its weight fragments stay in registers (wpre)
  // for the whole launch: the same fragments serve every step
  const int nks = dh / 32;
  int gu = -1, gk0 = 0, gk1 = nks;
  if (NG >= NW) {
    if (wave < NG) gu = wave;
  } else if (wave < NG * (NW / NG)) {
    const int WPG = NW / NG, f = wave / NG;
    gu = wave % NG;
    gk0 = (nks * f) / WPG;
    gk1 = (nks * (f + 1)) / WPG;
  }
  typename Gates<TW>::Pre wpre;
  const bool wkeep = !a.nocorr && Gates<TW>::kPre > 0 && use_pin && gu >= 0 &&
                     gk1 - gk0 <= Gates<TW>::kPre;
  // Domino's head: this wave's W_1^S fragments (rank tiles wave and wave + NW,
  // k groups q < UW / 16) stay in registers for the whole launch when they fit
  // (compile-time shapes only: elsewhere the registers are better spent)
  constexpr int kW1T = 2, kW1Q = 2;
  typename W4<TW>::T w1f[kW1T][kW1Q];
  const bool w1keep = HEAD && SDH > 0 && a.rank / 16 <= kW1T * NW && UW / 16 <= kW1Q;
  // ---- the candidates: every known node scoring >= vB, the B-th best known
  // score -- the only nodes that can still be popped or expanded.  They stay
  // listed in one of two buffers (S_CLIST names it, S_NCAND their number); a
  // step ranks the old candidates and its new children, which all scored >=
  // the old vB when they were appended; no other node can be among the B
  // best.  A value is a candidate when fewer than B values exceed it.  Both
  // rankings write the next list (S_NNEXT0 + npar entries, with the scores of the
  // first kCsCap) and each wave's least candidate score (S_CNT0 + wave); the
  // select step then sets vB from them.
  //
  // rank_list: the current list holds nval entries, candidates then children,
  // with their scores; a child's code becomes its table index, base + xoff[c]
  // + rank (xoff: this wave's own copy of the offsets, written before the
  // call).
  int npar = 0;     // S_NNEXT0 + npar counts the next list (the same in every wave)
  int clist_r = 0;  // the current list (S_CLIST; the same in every wave)
  auto rank_list = [&](int clist, int nval, int base) {
    const float *cv = clist ? cs2 : cs;
    const int16_t *ci = clist ? elist2 : elist;
    float *nv = clist ? cs : cs2;
    int16_t *ni = clist ? elist : elist2;
    const float4 *c4 = reinterpret_cast<const float4 *>(cv);
    const int n4 = nval >> 2, t0 = n4 * 4;
    float best = __builtin_huge_valf();
    for (int q = tid; q < nval; q += NT) {
      const float gi = cv[q];
      int cnt = 0;
#pragma unroll 4
      for (int j = 0; j < n4; ++j) {  // (no early exit: the loads stay in flight together)
        const float4 v = c4[j];
        cnt += (v.x > gi) + (v.y > gi) + (v.z > gi) + (v.w > gi);
      }
      // the last nval % 4 entries (read together; entries past nval are not counted)
      const float e0 = cv[min(t0, kCsCap - 1)], e1 = cv[min(t0 + 1, kCsCap - 1)],
                  e2 = cv[min(t0 + 2, kCsCap - 1)];
      cnt += (t0 < nval && e0 > gi) + (t0 + 1 < nval && e1 > gi) + (t0 + 2 < nval && e2 > gi);
      if (cnt < B) {  // among the B best (ties included): a candidate
        best = fminf(best, gi);
        int id = ci[q];
        if (id < 0) {
          const int e = -1 - id;
          id = base + xoff[e >> 8] + (e & 255);
        }
        const int j = atomicAdd(&scal[S_NNEXT0 + npar], 1);
        ni[j] = (int16_t)id;
        if (j < kCsCap) nv[j] = gi;
      }
    }
    best = wave_min_f(best);
    if (lane == 0) scalf[S_CNT0 + wave] = best;
  };
  // rank_table: the old candidates and the nodes appended since the last
  // ranking (from S_ABASE) are gathered and ranked, or, if more than the
  // gather buffer holds, every node of the table.
  const int kGather = CH * MP;  // floats of `ell`, free between expansion steps
  auto rank_table = [&]() {
    const int nn = scal[S_NN];
    const int ncand = scal[S_NCAND];
    const int abase = scal[S_ABASE];
    const int clist = clist_r;
    const int16_t *cur = clist ? elist2 : elist;
    int16_t *nxt = clist ? elist : elist2;
    float *nv = clist ? cs : cs2;
    const int ntot = ncand + (nn - abase);
    const bool incr = ntot <= kGather;
    const int nr = incr ? ntot : nn;  // nodes ranked
    float *cg = ell;
    if (incr)
      for (int q = tid; q < ntot; q += NT) cg[q] = ng[q < ncand ? cur[q] : abase + q - ncand];
    __syncthreads();
    const float *src = incr ? cg : ng;
    const float4 *g4 = reinterpret_cast<const float4 *>(src);
    const int n4 = nr >> 2;
    float best = __builtin_huge_valf();
    for (int q = tid; q < nr; q += NT) {
      const float gi = src[q];
      int cnt = 0;
#pragma unroll 4
      for (int j = 0; j < n4; ++j) {
        const float4 v = g4[j];
        cnt += (v.x > gi) + (v.y > gi) + (v.z > gi) + (v.w > gi);
      }
      for (int j = n4 * 4; j < nr; ++j) cnt += src[j] > gi;
      if (cnt < B) {
        best = fminf(best, gi);
        const int j = atomicAdd(&scal[S_NNEXT0 + npar], 1);
        nxt[j] = (int16_t)(incr ? (q < ncand ? cur[q] : abase + q - ncand) : q);
        if (j < kCsCap) nv[j] = gi;
      }
    }
    best = wave_min_f(best);
    if (lane == 0) scalf[S_CNT0 + wave] = best;
  };

  int pb = 0;  // partial-buffer parity
  // L2 prefetches of the next staging's rows, consumed after its wait
  float pf[3] = {0.0f, 0.0f, 0.0f};
  auto expand_chunk = [&](const int16_t *cn, int nc, int d) {
    // one batched round trip: the merged row of depth d (the children's
    // candidates and tail) and the parent path states of the chunk's nodes
    const int32_t *ccand = rcand;
    const float *ccandv = rcandv;
    // (this wave's W_hh fragments, when they fit kPre k steps, are in wpre:
    // loaded once before the first step and kept in registers)
    const bool wearly = wkeep && d > 0;
    // the root with no h0: its state is zero, so U . S = 0 and the correction is
    // the E[v] . b_c the row merge already added -- no exchange
    // (Domino's head is not zero at a zero state: SiLU(a_d))
    const bool nocorr = a.nocorr || (!HEAD && d == 0 && a.h0 == nullptr);
    if (d > 0 && tid < nc) nstate[cn[tid]] = (int16_t)(scal[S_NEXP] + tid);
    // the chunk's nodes in registers (lane c < nc of every wave): node, token,
    // score and the parent's state slot, read once; the new state of node c
    // goes to slot q_base + c
    const int root_slot = a.ecap - 1;
    const int q_base = scal[S_NEXP];
    int q_node = 0, q_tok = 0, q_pslot = root_slot;
    float q_g = 0.0f;
    if (d > 0 && lane < nc) {
      q_node = cn[lane];
      q_tok = ntok[q_node];
      q_g = ng[q_node];
      const int par = nparent[q_node];
      if (par >= 0) q_pslot = nstate[par];
    }
    {
      // all loads are issued before the first LDS write (one wait)
      const size_t row = (size_t)t * L + (d < L ? d : 0);
      const __amdgpu_buffer_rsrc_t rc = dev_rsrc(a.cand + row * M);
      const __amdgpu_buffer_rsrc_t rv = dev_rsrc(a.candv + row * M);
      const __amdgpu_buffer_rsrc_t rs = dev_rsrc(a.states + (size_t)t * a.ecap * dh);
      const bool rowld = d < L && tid < M;
      int32_t cid = 0;
      float cval = NEG_INF, rt = NEG_INF;
      if (rowld) {
        cid = __builtin_bit_cast(int32_t, ld_dev4(rc, tid * 4));
        cval = ld_dev4(rv, tid * 4);
      }
      if (d < L && tid == NT - 1) rt = ld_dev(a.tailR + row);
      // parent states straight into LDS (16 bytes per lane, 256 floats per
      // wave instruction), the chunk's nc columns only: the MFMA outputs of the
      // other columns are never read (an instruction that reaches past column
      // nc - 1 reads the root slot there)
      if (d > 0 && !a.nocorr) {
        for (int i = wave; i < (nc * dh + 255) / 256; i += NW) {
          const int e = i * 256 + 4 * lane;
          const int c = e / dh, k = e - c * dh;
          const int slot = __builtin_amdgcn_ds_bpermute(c * 4, q_pslot);  // (root slot for c >= nc)
          // (one row, or whole rows when unpadded: the 256 floats are contiguous)
          const int c0 = (i * 256) / dh;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              rs, (__attribute__((address_space(3))) void *)(Sp + c0 * SPS + (i * 256 - c0 * dh)),
              16, (slot * dh + k) * 4, 0, 0, kSc1);
        }
      }
      // this member's U slice of depth d's candidates, straight into LDS
      if (a.use_us && d < L && !nocorr) {
        const __amdgpu_buffer_rsrc_t ru =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(a.U_all), 0, 0x7FFFFFF0, 0x00020000);
        for (int i = wave; i < MP * UW / 256; i += NW) {
          const int e = i * 256 + 4 * lane;
          const int m = e / UW, k = e - m * UW;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              ru, (__attribute__((address_space(3))) void *)(Us + i * 256), 16,
              (rowids[d * MP + m] * dh + member * UW + k) * 4, 0, 0, 0);
        }
      }
      // Domino's head: this member's rank slice of the W_2 rows of depth d's
      // candidates straight into LDS (16 bytes per lane, lpr lanes per row),
      // and of the depth's a_d
      float hav = 0.0f;
      if constexpr (HEAD) {
        if (d < L) {
          const int es = (int)sizeof(TW);
          const int lpr = a.RJ * es / 16;  // lanes per row
          const __amdgpu_buffer_rsrc_t rw2 =
              __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(a.w2), 0, 0x7FFFFFF0, 0x00020000);
          for (int i = wave; i < MP * lpr / 64; i += NW) {
            const int m = i * (64 / lpr) + lane / lpr, part = lane - (lane / lpr) * lpr;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rw2, (__attribute__((address_space(3))) void *)(hw2 + i * 1024), 16,
                (rowids[d * MP + m] * a.rank + member * a.RJ) * es + part * 16, 0, 0, 0);
          }
          if (tid < a.RJ) hav = a.ha[((size_t)t * L + d) * a.rank + member * a.RJ + tid];
        }
      }
      // GRU inputs of the chunk's nodes straight into LDS, one wave instruction
      // per node: lane l < 3 UW/4 takes 4 floats of gate l / (UW/4); the other
      // lanes re-read the first 16 bytes into the slot's unused tail
      if (use_pin && d > 0 && !a.nocorr) {
        const int QW = UW / 4;
        const int g = lane / QW, k = (lane - g * QW) * 4;
        const int voff = lane < 3 * QW ? (g * dh + k) * 4 : 0;
        for (int c = wave; c < nc; c += NW) {
          const int tok = __builtin_amdgcn_readlane(q_tok, c);
          const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc(
              const_cast<float *>(a.P_all + (size_t)tok * (3 * dh) + member * UW), 0, 0x7FFFFFF0,
              0x00020000);
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              rp, (__attribute__((address_space(3))) void *)(pin + c * kPinSlot), 16, voff, 0, 0, 0);
        }
      }
      if (tid < MP) {
        rcand[tid] = rowld ? cid : 0;
        rcandv[tid] = rowld ? cval : NEG_INF;
      }
      if (tid == NT - 1) scalf[S_R] = rt;
      __builtin_amdgcn_s_waitcnt(0);  // includes the LDS writes of the loads above
      asm volatile("" ::"v"(pf[0]), "v"(pf[1]), "v"(pf[2]));  // (the prefetches: done)
      if (HEAD && tid < a.RJ) has[tid] = hav;
    }
    __syncthreads();
    // 1. path states of this member's units: S = GRU(S_parent, E[token]) (section 2.3)
    if (nocorr) {
      // (no path states without the correction)
    } else if (d == 0) {
      for (int u = tid; u < UW; u += NT) {
        const int j = member * UW + u;
        for (int c = 0; c < CH; ++c) Sn[c * UW + u] = (c == 0 && a.h0) ? a.h0[(size_t)t * dh + j] : 0.0f;
      }
    } else {
      const int c = lane & 15;
      const int node = c < nc ? cn[c] : -1;
      const float *prow = use_pin ? a.P_all : a.P_all + (size_t)(node >= 0 ? ntok[node] : 0) * (3 * dh);
      // r = sig(P_r + W_hr h), z = sig(P_z + W_hz h), n = tanh(P_n + r (W_hn h + b_hn)),
      // S = (1 - z) n + z h  (P_r, P_z carry b_hr, b_hz)
      auto apply = [&](int gi, const f32x4 (&gh)[3]) {
        if (node < 0) return;
        const int u4 = gi * 16 + (lane >> 4) * 4;  // first of this lane's 4 units (in the member)
        const int j0 = member * UW + u4;
        GruIn in;
        if (use_pin) {
          const float *pr = pin + c * kPinSlot + u4;
          in.r = *reinterpret_cast<const float4 *>(pr);
          in.z = *reinterpret_cast<const float4 *>(pr + UW);
          in.n = *reinterpret_cast<const float4 *>(pr + 2 * UW);
          in.b = *reinterpret_cast<const float4 *>(bhn + u4);
        } else {
          in = load_gru_in(prow, a.b_hh, dh, j0);
        }
        const float xr[4] = {in.r.x, in.r.y, in.r.z, in.r.w}, xz[4] = {in.z.x, in.z.y, in.z.z, in.z.w};
        const float xn[4] = {in.n.x, in.n.y, in.n.z, in.n.w}, xb[4] = {in.b.x, in.b.y, in.b.z, in.b.w};
        float sv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float r = sigmoid_fast(xr[i] + gh[0][i]);
          const float z = sigmoid_fast(xz[i] + gh[1][i]);
          const float n = tanh_fast(xn[i] + r * (gh[2][i] + xb[i]));
          const float hprev = Sp[c * SPS + j0 + i];
          sv[i] = (1.0f - z) * n + z * hprev;
          Sn[c * UW + u4 + i] = sv[i];
        }
        const __amdgpu_buffer_rsrc_t rsw = dev_rsrc(a.states + (size_t)t * a.ecap * dh);
        st_dev16(rsw, ((q_base + c) * dh + j0) * 4, make_float4(sv[0], sv[1], sv[2], sv[3]));
      };
      if (NG >= NW) {
        for (int gi = wave; gi < NG; gi += NW) {
          f32x4 gh[3];
          if (wearly && gi == wave)
            Gates<TW>::run_pre(a, Sp, wpre, 0, nks, gh);
          else
            Gates<TW>::run(a, Sp, u0 + gi, 0, nks, gh);
          apply(gi, gh);
        }
      } else {
        // WPG waves split the k range of one unit group; partial sums meet in LDS
        const int WPG = NW / NG;
        if (wave < NG * WPG) {
          f32x4 gh[3];
          if (wearly)
            Gates<TW>::run_pre(a, Sp, wpre, gk0, gk1, gh);
          else
            Gates<TW>::run(a, Sp, u0 + gu, gk0, gk1, gh);
#pragma unroll
          for (int g = 0; g < 3; ++g)
#pragma unroll
            for (int i = 0; i < 4; ++i) gpart[((wave * 3 + g) * 64 + lane) * 4 + i] = gh[g][i];
        }
        __syncthreads();
        // gate sums and the update, one (unit, node) per thread: element e holds
        // MFMA output lane l = (e / 4) % 64, row i = e % 4 of unit group e / 256,
        // i.e. node l % 16 and unit 16 (e / 256) + 4 (l / 16) + i.  The four
        // lanes of a quad hold four consecutive units of one node: the first
        // stores them with one 16-byte store.
        const __amdgpu_buffer_rsrc_t rsw = dev_rsrc(a.states + (size_t)t * a.ecap * dh);
        for (int e0 = 0; e0 < NG * 256; e0 += NT) {
          const int e = e0 + tid;
          const int gi = e >> 8, l = (e >> 2) & 63, i = e & 3;
          const int cc = l & 15;
          const bool live = e < NG * 256 && cc < nc;  // uniform over a quad
          const int u = gi * 16 + (l >> 4) * 4 + i;
          const int j = member * UW + u;
          float sv = 0.0f;
          if (live) {
            float gs[3];
#pragma unroll
            for (int g = 0; g < 3; ++g) {
              float sum = 0.0f;
              for (int ff = 0; ff < WPG; ++ff) sum += gpart[(((ff * NG + gi) * 3 + g) * 64 + l) * 4 + i];
              gs[g] = sum;
            }
            float xr, xz, xn, xb;
            if (use_pin) {
              const float *pr = pin + cc * kPinSlot + u;
              xr = pr[0];
              xz = pr[UW];
              xn = pr[2 * UW];
              xb = bhn[u];
            } else {
              // buffer loads: a pointer shared with the LDS branch would make
              // both flat accesses
              const __amdgpu_buffer_rsrc_t rpr = __builtin_amdgcn_make_buffer_rsrc(
                  const_cast<float *>(a.P_all + (size_t)ntok[cn[cc]] * (3 * dh)), 0, 0x7FFFFFF0, 0x00020000);
              const __amdgpu_buffer_rsrc_t rbh =
                  __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(a.b_hh), 0, 0x7FFFFFF0, 0x00020000);
              xr = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rpr, j * 4, 0, 0));
              xz = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rpr, (dh + j) * 4, 0, 0));
              xn = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rpr, (2 * dh + j) * 4, 0, 0));
              xb = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rbh, (2 * dh + j) * 4, 0, 0));
            }
            const float r = sigmoid_fast(xr + gs[0]);
            const float z = sigmoid_fast(xz + gs[1]);
            const float n = tanh_fast(xn + r * (gs[2] + xb));
            sv = (1.0f - z) * n + z * Sp[cc * SPS + j];
            Sn[cc * UW + u] = sv;
          }
          const float s1 = sel::dpp_f<0x55>(sv), s2 = sel::dpp_f<0xAA>(sv), s3 = sel::dpp_f<0xFF>(sv);
          if (live && i == 0) st_dev16(rsw, ((q_base + cc) * dh + j) * 4, make_float4(sv, s1, s2, s3));
        }
      }
    }
    __syncthreads();
    if (d >= L) return;
    // 2. this member's part of delta[c][m] = U[cand[m]] . S_c over its units (fp32 MFMA)
    const int RT = (M + 15) / 16;
    const int nq = UW / 16;
    // parts of member j: a [CH][MP] block of their own (no line is shared by two writers)
    const __amdgpu_buffer_rsrc_t rmy =
        dev_rsrc(a.part + (((size_t)t * 2 + pb) * G + member) * CH * MP);
    if constexpr (HEAD) {
      // Domino's head (section 2.3).  (a) this member's part of W_1^S S_c over
      // its units, 16 ranks per MFMA tile, published for the other members.
      // The exchange is reader-major: [reader j][writer][node c][RJ ranks], so
      // the parts member j sums are one contiguous block of blk floats
      const int RJ = a.RJ, RJ4 = RJ / 4, blk = G * CH * RJ;
      const size_t tp = ((size_t)t * 2 + pb) * G * blk;
      const __amdgpu_buffer_rsrc_t rhp = dev_rsrc(a.hpart + tp + member * CH * RJ);
      const int c = lane & 15, kq = (lane >> 4) * 4;
      auto mma4 = [&](f32x4 acc, float4 av, float4 bv) {
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.x, bv.x, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.y, bv.y, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.z, bv.z, acc, 0, 0, 0);
        return __builtin_amdgcn_mfma_f32_16x16x4f32(av.w, bv.w, acc, 0, 0, 0);
      };
      // lane l, register i of a tile: rank rt*16 + (l/16)*4 + i of node l%16
      // (the four ranks of a lane share one reader: RJ % 16 == 0)
      auto publish = [&](int rt, f32x4 acc) {
        if (c < nc) {
          const int r = rt * 16 + (lane >> 4) * 4, j = r / RJ;
          st_dev16(rhp, (j * blk + c * RJ + r - j * RJ) * 4, make_float4(acc[0], acc[1], acc[2], acc[3]));
        }
      };
      if (w1keep) {
#pragma unroll
        for (int j = 0; j < kW1T; ++j) {
          const int rt = wave + j * NW;
          if (rt < a.rank / 16) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < kW1Q; ++q)
              if (q < nq)
                acc = mma4(acc, W4<TW>::widen(w1f[j][q]),
                           *reinterpret_cast<const float4 *>(Sn + c * UW + q * 16 + kq));
            publish(rt, acc);
          }
        }
      } else {
        for (int rt = wave; rt < a.rank / 16; rt += NW) {
          const TW *w1r = static_cast<const TW *>(a.w1) + (size_t)(rt * 16 + c) * a.ld1 + a.d_H + member * UW;
          f32x4 acc = {0.f, 0.f, 0.f, 0.f};
          for (int q = 0; q < nq; ++q)
            acc = mma4(acc, load4w(w1r + q * 16 + kq),
                       *reinterpret_cast<const float4 *>(Sn + c * UW + q * 16 + kq));
          publish(rt, acc);
        }
      }
      group_barrier(ctr, G, nbar, &scal[S_STATUS], a.spin_limit);
      if (scal[S_STATUS] & DT_TREE_TIMEOUT) return;  // (uniform: read after the barrier)
      // (b) this member's rank slice of y = SiLU(a_d + W_1^S S) for the chunk's
      // nodes.  An item is (node c, 4 ranks); P lanes of one wave share an item,
      // each summing every P-th member's part, then a butterfly over the P lanes
      // (the same sum in every lane: deterministic).  Columns c >= nc of y are
      // not read back: their MFMA outputs are dropped.
      {
        const int P = G < 8 ? G : 8;  // (G is a power of two)
        const int sub = lane & (P - 1), nitem = nc * RJ4;
        const __amdgpu_buffer_rsrc_t rha = dev_rsrc(a.hpart + tp + (size_t)member * blk);
        for (int e0 = wave * (64 / P); e0 < nitem; e0 += NW * (64 / P)) {  // (wave-uniform)
          const int e = e0 + lane / P;
          float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
          if (e < nitem)
            for (int m2 = sub; m2 < G; m2 += P) sum += ld_dev16(rha, (m2 * CH * RJ + e * 4) * 4);
          for (int o = 1; o < P; o <<= 1) {
            sum.x += __shfl_xor(sum.x, o);
            sum.y += __shfl_xor(sum.y, o);
            sum.z += __shfl_xor(sum.z, o);
            sum.w += __shfl_xor(sum.w, o);
          }
          if (e < nitem && sub == 0) {
            const int cc = e / RJ4, r4 = (e - cc * RJ4) * 4;  // e * 4 = cc * RJ + r4
            const float x[4] = {has[r4] + sum.x, has[r4 + 1] + sum.y, has[r4 + 2] + sum.z,
                                has[r4 + 3] + sum.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) hys[cc * RJ + r4 + i] = x[i] * sigmoid_fast(x[i]);
          }
        }
      }
      __syncthreads();
      // (c) this member's part of delta[c][m] = W_2[cand_m] . y over its rank slice
      for (int rt = wave; rt < RT; rt += NW) {
        const TW *w2row = reinterpret_cast<const TW *>(hw2) + (rt * 16 + c) * RJ;  // slots >= M: unused
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        for (int q = 0; q < RJ / 16; ++q)
          acc = mma4(acc, load4w(w2row + q * 16 + kq),
                     *reinterpret_cast<const float4 *>(hys + c * RJ + q * 16 + kq));
        // (lane l, register i: slot rt*16 + (l/16)*4 + i of node l%16)
        if (c < nc)
          st_dev16(rmy, (c * MP + rt * 16 + (lane >> 4) * 4) * 4,
                   make_float4(acc[0], acc[1], acc[2], acc[3]));
      }
    }
    // (two instances of the loop, the U rows from the LDS slice or from
    // memory: one load instruction serving both would be a flat load, whose
    // wait also waits for the state stores just issued)
    auto corr_tiles = [&](auto from_lds) {
      constexpr bool LDSU = decltype(from_lds)::value;
      for (int rt = (nocorr || HEAD) ? RT : wave; rt < RT; rt += NW) {
        const int m = rt * 16 + (lane & 15);
        const int c = lane & 15, kq = (lane >> 4) * 4;
        const float *urow = a.U_all + (size_t)(m < M ? ccand[m] : 0) * dh + member * UW;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        for (int q = 0; q < nq; ++q) {
          float4 av = make_float4(0.f, 0.f, 0.f, 0.f);
          if constexpr (LDSU)
            av = *reinterpret_cast<const float4 *>(Us + m * UW + q * 16 + kq);  // slots >= M: row 0, unused
          else if (m < M)
            av = *reinterpret_cast<const float4 *>(urow + q * 16 + kq);
          const float4 bv = *reinterpret_cast<const float4 *>(Sn + c * UW + q * 16 + kq);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.x, bv.x, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.y, bv.y, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.z, bv.z, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.w, bv.w, acc, 0, 0, 0);
        }
        // lane l, register i: slot rt*16 + (l/16)*4 + i, node l%16
        if (c < nc)
          st_dev16(rmy, (c * MP + rt * 16 + (lane >> 4) * 4) * 4,
                   make_float4(acc[0], acc[1], acc[2], acc[3]));
      }
    };
    if (a.use_us)
      corr_tiles(std::true_type{});
    else
      corr_tiles(std::false_type{});
    if (!nocorr) group_barrier(ctr, G, nbar, &scal[S_STATUS], a.spin_limit);
    if (scal[S_STATUS] & DT_TREE_TIMEOUT) return;  // (uniform: read after the barrier)
    // 3. children of each node: normalise, rank, keep the top-k above vB
    const float vB = scalf[S_VB];
    const float R = scalf[S_R];
    const int clist = clist_r;  // the candidate list the children join
    const __amdgpu_buffer_rsrc_t rp = dev_rsrc(a.part + ((size_t)t * 2 + pb) * G * CH * MP);
    pb ^= 1;
    // the G parts of a slot, one from each member's block: all loads are
    // issued, then summed in member order
    auto load_parts = [&](int c, int s) -> Parts {
      Parts p;
      const int r = lane >> 4, stride = CH * MP * 4;
      const int off = (c * MP + 64 * s + 4 * (lane & 15)) * 4 + r * stride;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p.v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        // (the stride of four members goes in the scalar offset)
        if (4 * i + r < G) p.v[i] = ld_dev16(rp, off, 4 * i * stride);
      }
      return p;
    };
    auto node_children = [&](int c, const Parts &p0) -> int {
      const float gpar = (d == 0) ? 0.0f : __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, q_g), c));
      float lv[4];
      if (a.menu_in) {
        // a shared menu: depth d's slot log-probs, already normalised
        const float *mrow = a.menu_in + ((size_t)t * L + d) * MP;
#pragma unroll
        for (int s = 0; s < 4; ++s)
          if (s < MP / 64) lv[s] = mrow[lane + 64 * s];
      } else {
        float zv[4];
        float mx = NEG_INF;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          if (s >= MP / 64) break;
          const int m = lane + 64 * s;
          // x already holds logit + E[v] . b_c (added by the row merge; not for the marginals)
          const float x = ccandv[m];
          const float dl = nocorr ? x : x + sum_parts(s == 0 ? p0 : load_parts(c, s), lane);
          const float z = x > NEG_INF ? dl * a.inv_tau : NEG_INF;  // slots >= M hold -inf
          zv[s] = z;
          mx = fmaxf(mx, z);
        }
        mx = wave_max_f(mx);
        const bool tail = (a.norm_mode == DT_NORM_TAIL) && R > NEG_INF;
        if (tail) mx = fmaxf(mx, R);
        float sum = 0.0f;
#pragma unroll
        for (int s = 0; s < 4; ++s)
          if (s < MP / 64) sum += (zv[s] > NEG_INF) ? exp_hw(zv[s] - mx) : 0.0f;
        sum = wave_sum_f(sum);
        if (tail) sum += exp_hw(R - mx);
        const float logZ = mx + log_hw(sum);
#pragma unroll
        for (int s = 0; s < 4; ++s)
          if (s < MP / 64) lv[s] = (zv[s] > NEG_INF) ? zv[s] - logZ : NEG_INF;
      }
      if (a.menu_out && member == 0) {
        // this node's slot log-probs: depth d's menu (one node per depth in a chain)
        float *mrow = a.menu_out + ((size_t)t * L + d) * MP;
#pragma unroll
        for (int s = 0; s < 4; ++s)
          if (s < MP / 64) mrow[lane + 64 * s] = lv[s];
      }
      // E: the slots whose child could enter (log-prob finite, g >= vB).  A slot
      // ranked above a member of E is in E itself, so a member's rank among
      // all slots is its rank within E.
      uint64_t em[4];
      int ne = 0;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        em[s] = 0ull;
        if (s >= MP / 64) break;
        em[s] = __ballot(lv[s] > NEG_INF && gpar + lv[s] >= vB);
        ne += __popcll(em[s]);
        ell[c * MP + lane + 64 * s] = lv[s];
      }
      if (ne == 0) {
        if (lane == 0) wcnt[c] = 0;
        return 0;
      }
      int kc = 0;
      if (ne <= 24) {
        // few members: walk E's slots, (log-prob desc, slot asc)
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          if (s >= MP / 64) break;
          const int m = lane + 64 * s;
          const float lm = lv[s];
          int rank = 0;
#pragma unroll
          for (int s2 = 0; s2 < 4; ++s2) {
            if (s2 >= MP / 64) break;
            uint64_t b = em[s2];
            while (b) {
              const int bl = __builtin_ctzll(b);
              b &= b - 1;
              const float l2 = __builtin_bit_cast(
                  float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, lv[s2]), bl));
              rank += (l2 > lm) | ((l2 == lm) & (64 * s2 + bl < m));
            }
          }
          const bool keep = ((em[s] >> lane) & 1ull) && rank < a.k;
          kc += __popcll(__ballot(keep));
          rnk[c * MP + m] = keep ? (int16_t)rank : (int16_t)-1;
        }
      } else if (MP == 64) {
        // many members (the root while vB is -inf): one bitonic sort of E's keys,
        // (log-prob desc, slot asc); lane j of the sorted keys holds rank j
        const uint64_t srt = sel::wave_sort64(
            ((em[0] >> lane) & 1ull) ? make_key(lv[0], (uint32_t)lane) : 0ull, true);
        const bool keep = srt != 0ull && lane < a.k;
        rnk[c * MP + lane] = (int16_t)-1;
        if (keep) rnk[c * MP + (int)key_index(srt)] = (int16_t)lane;
        kc = __popcll(__ballot(keep));
      } else {
        wave_sync();
        const float4 *e4 = reinterpret_cast<const float4 *>(ell + c * MP);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          if (s >= MP / 64) break;
          const int m = lane + 64 * s;
          const float lm = lv[s];
          // rank = slots ahead of m by (log-prob desc, slot asc); slots >= M hold -inf
          int rank = 0;
#pragma unroll 4
          for (int q = 0; q < MP / 4; ++q) {
            const float4 v = e4[q];
            const int m2 = 4 * q;
            rank += (v.x > lm) | ((v.x == lm) & (m2 < m));
            rank += (v.y > lm) | ((v.y == lm) & (m2 + 1 < m));
            rank += (v.z > lm) | ((v.z == lm) & (m2 + 2 < m));
            rank += (v.w > lm) | ((v.w == lm) & (m2 + 3 < m));
          }
          const bool keep = ((em[s] >> lane) & 1ull) && rank < a.k;
          kc += __popcll(__ballot(keep));
          rnk[c * MP + m] = keep ? (int16_t)rank : (int16_t)-1;
        }
      }
      if (lane == 0) wcnt[c] = kc;
      return kc;
    };
    // two nodes per wave: the second node's loads are in flight during the first
    const int c0 = wave, c1 = wave + NW;
    Parts p0, p1;
    if (c0 < nc && !nocorr) p0 = load_parts(c0, 0);
    if (c1 < nc && !nocorr) p1 = load_parts(c1, 0);
    int k0 = 0, k1 = 0;
    if (c0 < nc)
      k0 = node_children(c0, p0);
    else if (lane == 0)
      wcnt[c0] = 0;
    if (c1 < nc)
      k1 = node_children(c1, p1);
    else if (lane == 0)
      wcnt[c1] = 0;
    // The kept children also join this step's candidate list after the old
    // candidates (positions from one counter per wave; their order does not
    // matter): score, and the code -1 - (256 c + rank), which becomes a table
    // index once the nodes' offsets are known.  Entries past kCsCap are
    // dropped (the step then ranks the table instead).  Ranks and log-probs
    // are read back from this wave's own rnk and ell rows.
    if (k0 + k1 > 0) {
      int o = 0;
      if (lane == 0) o = atomicAdd(&scal[S_NVAL], k0 + k1);
      o = __builtin_amdgcn_readlane(o, 0);
      float *lcs = clist ? cs2 : cs;
      int16_t *lci = clist ? elist2 : elist;
      for (int h = 0; h < 2; ++h) {
        const int c = h ? c1 : c0, oc = h ? o + k0 : o;
        if ((h ? k1 : k0) == 0) continue;
        const float gpar = (d == 0) ? 0.0f : __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, q_g), c));
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          if (s >= MP / 64) break;
          const int m = lane + 64 * s;
          const int r = rnk[c * MP + m];
          if (r >= 0 && oc + r < kCsCap) {
            lcs[oc + r] = gpar + ell[c * MP + m];
            lci[oc + r] = (int16_t)(-1 - (c * 256 + r));
          }
        }
      }
    }
    // (read before the barrier: thread 0 rewrites it after the barrier)
    const int base = scal[S_NN];
    __syncthreads();
    // 4. append children (node order, then rank order) to the node table: node
    // c's children start at base + the children of nodes 0..c-1 (a prefix sum
    // over the lanes of row 0; nc <= 16)
    const int wc = lane < nc ? wcnt[lane] : 0;
    const int nval = scal[S_NVAL];
    const int incl = row_prefix16(wc);
    const int tot = __builtin_amdgcn_readlane(incl, 15);
    const int excl = incl - wc;
    // (every wave writes the same offsets; each reads back its own)
    if (lane < CH) xoff[lane] = excl;
    for (int c = wave; c < nc; c += NW) {
      if (__builtin_amdgcn_readlane(wc, c) == 0) continue;
      const int off = base + __builtin_amdgcn_readlane(excl, c);
      const float gpar = (d == 0) ? 0.0f : __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, q_g), c));
      #pragma unroll
      for (int s = 0; s < 4; ++s) {
        if (s >= MP / 64) break;
        const int m = lane + 64 * s;
        const int rk = m < M ? rnk[c * MP + m] : -1;
        if (rk >= 0) {
          const int pos = off + rk;
          if (pos < NC) {
            ng[pos] = gpar + ell[c * MP + m];
            ntok[pos] = ccand[m];
            nslot[pos] = (int16_t)m;
            ndepth[pos] = (uint8_t)(d + 1);
            nparent[pos] = (d == 0) ? (int16_t)-1 : (int16_t)__builtin_amdgcn_readlane(q_node, c);
            nrank[pos] = (uint8_t)rk;
            nstate[pos] = -1;
            nexp[pos] = 0;
          }
        }
      }
    }
    // Prefetch into L2 what the next steps stage: the P rows (this member's
    // three gate slices, 128-byte lines) of the children this wave appended --
    // tokens read back from its own table writes -- and this member's U slice
    // of the next depth's candidates.  The values are consumed only after the
    // next staging's wait, so nothing waits for them earlier: their HBM latency
    // passes during the ranking and the select step.
    if (!a.nocorr) {
      const int LPS = (UW * 4 + 127) / 128;  // lines per gate slice
      const int per = 3 * LPS;               // lines per child
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int c = wave + h * NW;
        pf[h] = 0.0f;
        if (c < nc) {
          const int r = lane / per;
          const int pos = base + __builtin_amdgcn_readlane(excl, c) + r;
          if (r < __builtin_amdgcn_readlane(wc, c) && pos < NC) {
            const int gl = lane - r * per, g = gl / LPS;
            pf[h] = a.P_all[(size_t)ntok[pos] * (3 * dh) + g * dh + member * UW + (gl - g * LPS) * 32];
          }
        }
      }
      pf[2] = 0.0f;
      if (a.use_us && wave == NW - 1 && d + 1 < L) {
        const int m = lane / LPS;
        if (m < M)
          pf[2] = a.U_all[(size_t)rowids[(d + 1) * MP + m] * dh + member * UW + (lane - m * LPS) * 32];
      }
    }
    // 5. the candidates: rank the list of old candidates and new children in
    // place, or, when the table or the list overflowed, the table
    const bool inlist = base + tot <= NC && nval <= kCsCap;
    // (these writes touch no entry the appends above write)
    if (tid == 0) {
      int nn = base + tot;
      if (nn > NC) {
        nn = NC;
        scal[S_STATUS] |= DT_TREE_TRUNCATED;  // table overflow (massive exact ties)
      }
      scal[S_NN] = nn;
      scal[S_ABASE] = inlist ? nn : base;
      if (d > 0) scal[S_NEXP] += nc;
    }
    if (d > 0 && tid < nc) nexp[cn[tid]] = 1;
    if (inlist) {
      rank_list(clist, nval, base);
    } else {
      __syncthreads();
      rank_table();
    }
    __syncthreads();
  };

  // ---- drop the nodes below vB to make room (parents always score at least
  // their children, so the links stay valid); the candidate list is renumbered
  auto compact_table = [&]() {
    const int nn = scal[S_NN];
    const float vB = scalf[S_VB];
    for (int r0 = 0; r0 < nn; r0 += NT) {
      const int i = r0 + tid;
      const bool keep = i < nn && ng[i] >= vB;
      const Compact cp = block_compact(keep, wcnt);
      const int off = r0 ? scal[S_TOT] : 0;
      if (i < nn) newidx[i] = keep ? (int16_t)(cp.pos + off) : (int16_t)-1;
      __syncthreads();
      if (tid == 0) scal[S_TOT] = off + cp.total;
      __syncthreads();
    }
    const int kept = scal[S_TOT];
    constexpr int PER = (NC + NT - 1) / NT;
    float rg[PER];
    int rt_[PER], rp[PER], rs[PER], rsl[PER], rd[PER], rr[PER], re[PER], dst[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int i = tid + q * NT;
      dst[q] = (i < nn) ? newidx[i] : -1;
      if (dst[q] >= 0) {
        rg[q] = ng[i];
        rt_[q] = ntok[i];
        rp[q] = nparent[i] >= 0 ? newidx[nparent[i]] : -1;
        rs[q] = nstate[i];
        rsl[q] = nslot[i];
        rd[q] = ndepth[i];
        rr[q] = nrank[i];
        re[q] = nexp[i];
      }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      if (dst[q] >= 0) {
        const int j = dst[q];
        ng[j] = rg[q];
        ntok[j] = rt_[q];
        nparent[j] = (int16_t)rp[q];
        nstate[j] = (int16_t)rs[q];
        nslot[j] = (int16_t)rsl[q];
        ndepth[j] = (uint8_t)rd[q];
        nrank[j] = (uint8_t)rr[q];
        nexp[j] = (uint8_t)re[q];
      }
    }
    // every candidate scores >= vB, so it is kept
    int16_t *cur = scal[S_CLIST] ? elist2 : elist;
    const int ncand = scal[S_NCAND];
    for (int q = tid; q < ncand; q += NT) cur[q] = newidx[cur[q]];
    __syncthreads();
    if (tid == 0) {
      scal[S_NN] = kept;
      scal[S_ABASE] = kept;
    }
    __syncthreads();
  };

  // ---- phase A ---------------------------------------------------------------
  // Nodes enter the table in depth order (a chunk's children are one level
  // deeper than every node not yet reached), so one cursor walks it once: each
  // chunk is the next up-to-chunk_cap unexpanded nodes above depth L scoring
  // >= vB, all at the depth of the first of them.  A node the cursor passes
  // without taking scores below vB, and vB only grows, so it can never be
  // popped.
  if (wkeep) Gates<TW>::preload(a, u0 + gu, gk0, gk1, wpre);  // in flight while the loop starts
  if (w1keep) {
    const TW *w1m = static_cast<const TW *>(a.w1) + a.d_H + member * UW + (lane >> 4) * 4;
#pragma unroll
    for (int j = 0; j < kW1T; ++j)
#pragma unroll
      for (int q = 0; q < kW1Q; ++q) {
        const int rt = wave + j * NW;
        if (rt < a.rank / 16 && q < UW / 16)
          w1f[j][q] = W4<TW>::load(w1m + (size_t)(rt * 16 + (lane & 15)) * a.ld1 + q * 16);
      }
  }
  // One call site of expand_chunk (a second copy of the inlined step would
  // double the loop's code and its register shuffling): the first pass
  // expands the root (children at depth 1 scored from h0).
  int nsteps = 0;
  bool ranked = false;  // a ranking since the last select step
  int cur_r = 0;        // the cursor (the same in every wave)
  bool expand = true;   // a chunk to expand at the top of the loop
  int x_nc = 1, x_d = 0;
  for (;;) {
    if (expand) {
      expand_chunk(cl, x_nc, x_d);
      ranked = true;
      ++nsteps;
    }
    if (scal[S_STATUS] & DT_TREE_TIMEOUT) break;
    if (a.W > 0) {
      // Frontier builder (Appendix B): only the top W nodes of their depth, by
      // (score desc, table order), become lanes.  The table is depth-ordered,
      // and a depth's row is complete once the cursor reaches it (every node of
      // the depth above has been passed), which is when the flags are used.
      // Nodes the table dropped (below vB) rank below every node that can still
      // be taken, so counting the table gives the ledger's rank.
      const int nn = scal[S_NN];
      for (int i = tid; i < nn; i += NT) {
        const int di = ndepth[i];
        const float gi = ng[i];
        int r = 0;
        for (int j = i - 1; j >= 0 && ndepth[j] == di && r < a.W; --j) r += ng[j] >= gi;
        for (int j = i + 1; j < nn && ndepth[j] == di && r < a.W; ++j) r += ng[j] > gi;
        ins[i] = (uint8_t)(r < a.W);
      }
      __syncthreads();
    }
    // Every wave takes the select step itself, with identical results: vB,
    // the next list and the next chunk (the chunk and the shared words are
    // written with the same contents by every wave, and each reads back its
    // own), so no barrier follows it.  (The next step's staging barrier keeps
    // every wave's reads here ahead of the step's writes.)
    const int4 s0 = *reinterpret_cast<const int4 *>(scal);  // S_NN, S_VB, S_NEXP, S_STATUS
    const int nn = s0.x;
    float vB;
    if (ranked) {
      // vB from the ranking: the least candidate score, or -inf while fewer
      // than B nodes are known (every node is then a candidate); the next list
      // becomes the current one
      const float4 m0 = *reinterpret_cast<const float4 *>(scalf + S_CNT0);
      const float4 m1 = *reinterpret_cast<const float4 *>(scalf + S_CNT0 + 4);
      const int nnext = scal[S_NNEXT0 + npar];
      vB = fminf(fminf(fminf(m0.x, m0.y), fminf(m0.z, m0.w)), fminf(fminf(m1.x, m1.y), fminf(m1.z, m1.w)));
      if (nn < B) vB = -__builtin_huge_valf();
      clist_r ^= 1;
      if (lane == 0) {
        scalf[S_VB] = vB;
        scal[S_NCAND] = nnext;
        scal[S_CLIST] = clist_r;
        scal[S_ABASE] = nn;  // (a repeated ranking ranks no node twice)
        scal[S_NVAL] = nnext;
        scal[S_NNEXT0 + (npar ^ 1)] = 0;  // (read by every wave a ranking ago)
      }
      npar ^= 1;
    } else {
      vB = __builtin_bit_cast(float, s0.y);
    }
    int p = cur_r, c = 0, dsel = -1;
    bool done = false;
    while (!done && p < nn) {
      const int i = p + lane;
      const int ic = i < nn ? i : 0;  // (every load issued: one wait)
      const int ex = nexp[ic], dp = ndepth[ic], in_ = ins[ic];
      const float gg = ng[ic];
      const bool ok = (i < nn) & (ex == 0) & (dp < L) & (gg >= vB) & ((a.W == 0) | (in_ != 0));
      const int di = ok ? dp : -1;
      const uint64_t bal = __ballot(ok);
      if (bal == 0) {
        p += 64;
        continue;
      }
      if (dsel < 0) dsel = __builtin_amdgcn_readlane(di, __builtin_ctzll(bal));
      const uint64_t deeper = __ballot(ok && di != dsel);
      uint64_t use = __ballot(ok && di == dsel);
      if (deeper) use &= (1ull << __builtin_ctzll(deeper)) - 1;  // stop at the next depth
      const int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(use >> 32),
                                                   __builtin_amdgcn_mbcnt_lo((uint32_t)use, 0));
      const bool mine = (use >> lane) & 1ull;
      const int have = __popcll(use), need = chunk_cap - c;
      if (mine && before < need) cl[c + before] = (int16_t)i;
      if (have >= need) {
        // the cursor moves right past the need-th node taken
        const uint64_t last = __ballot(mine && before == need - 1);
        p += __builtin_ctzll(last) + 1;
        c = chunk_cap;
        done = true;
      } else {
        c += have;
        if (deeper) {
          p += __builtin_ctzll(deeper);
          done = true;
        } else {
          p += 64;
        }
      }
    }
    cur_r = p < nn ? p : nn;
    if (c && s0.z + c > a.ecap - 1) {
      if (tid == 0) atomicOr(&scal[S_STATUS], DT_TREE_TRUNCATED);
      break;
    }
    if (c == 0) break;
    int nc = c;
    if (nn + nc * a.k > NC - CH) {
      // make room for this chunk's children; the cursor restarts (nodes it
      // passed are expanded or below vB, and are passed again)
      __syncthreads();  // (every wave's select reads ahead of the moves)
      compact_table();
      if (tid == 0) {
        int c2 = 0;
        for (int c3 = 0; c3 < nc; ++c3) {
          const int i = newidx[cl[c3]];
          if (i >= 0) cl[c2++] = (int16_t)i;
        }
        scal[S_NC] = c2;
      }
      __syncthreads();
      nc = scal[S_NC];
      cur_r = 0;
    }
    ranked = false;
    expand = nc > 0;  // (none: select again)
    x_nc = nc;
    x_d = dsel;
  }
  // the last step's prefetches are waited for on the way out (after the
  // emission for the member that emits), not before the replay
  auto drain = [&]() {
    __builtin_amdgcn_s_waitcnt(0);
    asm volatile("" ::"v"(pf[0]), "v"(pf[1]), "v"(pf[2]));
  };
  if (scal[S_STATUS] & DT_TREE_TIMEOUT) {
    // a wait gave up: the tree may hold parts of members that had not written
    // them; it is emitted empty
    if (member == 0 && a.emit) emit_empty();
    drain();
    return;
  }
  if (a.stats && member == 0 && tid == 0) {
    a.stats[2 * t] = nsteps;
    a.stats[2 * t + 1] = scal[S_NEXP] + 1;  // the root and every expanded node
  }
  if (member != 0 || !a.emit) {
    drain();
    return;
  }

  // ---- phase B: exact replay of the heap --------------------------------------
  // Only nodes scoring >= vB (the B-th best score in the table) can be among
  // the first B pops: their ancestors score at least as much, so while fewer
  // than B have been popped one of them is always in the heap and outranks every
  // node below vB.  When at most 64 such nodes exist, one wave replays the heap
  // with a node per lane in registers; otherwise it scans the node table.
  // (vB is current: it is refreshed after every expansion step.)
  const int nn = scal[S_NN];
  if (a.W > 0) {
    // frontier builder: the ledger's global top B by (score desc, depth asc,
    // table order) -- a parent ranks before its children -- in that order
    const float vB = scalf[S_VB];
    for (int i = tid; i < nn; i += NT) {
      const float gi = ng[i];
      const int di = ndepth[i];
      int r = B;
      if (gi >= vB) {
        r = 0;
        for (int j = 0; j < nn && r < B; ++j) {
          const float gj = ng[j];
          r += (gj > gi) | ((gj == gi) & ((ndepth[j] < di) | ((ndepth[j] == di) & (j < i))));
        }
      }
      newidx[i] = (int16_t)(r < B ? r : -1);
      if (r < B) order[r] = (int16_t)i;
    }
    if (tid == 0) scal[S_NPOP] = 0;
    __syncthreads();
    int sel = 0;  // selected nodes this thread holds: min(B, nodes >= vB) in all
    for (int i = tid; i < nn; i += NT) {
      if (newidx[i] >= 0) {
        const int par = nparent[i];
        ppi[i] = (int16_t)(par >= 0 ? newidx[par] : -1);
        ++sel;
      }
    }
    if (sel) atomicAdd(&scal[S_NPOP], sel);
  } else if (wave == 0) {
    // the candidates (every node scoring >= vB) are listed, in any order
    const int ncand = scal[S_NCAND];
    const int16_t *clist = scal[S_CLIST] ? elist2 : elist;
    int npop = 0;
    bool done = false;
    if (ncand <= 64) {
      // Without exact score ties the pops are simply the candidates by score
      // (a parent scores strictly above its children, so it is popped first).
      const bool have = lane < ncand;
      const int me = have ? clist[lane] : -1;
      const float gm = have ? ng[me] : NEG_INF;
      Sn[lane] = gm;
      wave_sync();
      int rank = 0, eq = 0;
      const float4 *s4 = reinterpret_cast<const float4 *>(Sn);
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const float4 v = s4[q];
        rank += (v.x > gm) + (v.y > gm) + (v.z > gm) + (v.w > gm);
        eq += (v.x == gm) + (v.y == gm) + (v.z == gm) + (v.w == gm);
      }
      if (__ballot(have && eq > 1) == 0) {
        npop = ncand < B ? ncand : B;
        if (have) newidx[me] = (int16_t)rank;
        wave_sync();
        if (have && rank < B) {
          const int par = nparent[me];
          order[rank] = (int16_t)me;
          ppi[me] = (int16_t)(par >= 0 ? newidx[par] : -1);
        }
        done = true;
      }
    }
    if (!done && ncand <= 64) {
      const bool have = lane < ncand;
      const int me = have ? clist[lane] : -1;
      const int par = have ? nparent[me] : -2;
      const uint64_t gkey = have ? ((uint64_t)ordered_bits(ng[me]) << 32) |
                                       ((uint64_t)((~(uint32_t)nrank[me]) & 0xFFu) << 11) |
                                       (uint64_t)me
                                 : 0ull;
      bool ins_ = have && par < 0, popd_ = false;
      int ppi_ = -1;
      while (npop < B) {
        const uint64_t key =
            (ins_ && !popd_) ? gkey | ((uint64_t)((~(uint32_t)(ppi_ + 1)) & 0x1FFu) << 19) : 0ull;
        const uint64_t best = wave_max_u64(key);
        if (best == 0) break;
        const int p = (int)(best & 0x7FF);
        if (me == p) popd_ = true;
        if (par == p) {
          ins_ = true;
          ppi_ = npop;
        }
        if (lane == 0) order[npop] = (int16_t)p;
        ++npop;
      }
      if (have) ppi[me] = (int16_t)ppi_;
    } else if (!done) {
      for (int i = lane; i < nn; i += 64) {
        ins[i] = nparent[i] < 0;
        popd[i] = 0;
        ppi[i] = -1;
      }
      wave_sync();
      while (npop < B) {
        uint64_t best = 0;
        for (int i = lane; i < nn; i += 64) {
          if (ins[i] && !popd[i]) {
            const uint64_t key = ((uint64_t)ordered_bits(ng[i]) << 32) |
                                 ((uint64_t)((~(uint32_t)(ppi[i] + 1)) & 0x1FFu) << 19) |
                                 ((uint64_t)((~(uint32_t)nrank[i]) & 0xFFu) << 11) | (uint64_t)i;
            best = key > best ? key : best;
          }
        }
        best = wave_max_u64(best);
        if (best == 0) break;
        const int p = (int)(best & 0x7FF);
        if (lane == 0) {
          popd[p] = 1;
          order[npop] = (int16_t)p;
        }
        for (int i = lane; i < nn; i += 64)
          if (nparent[i] == p) {
            ins[i] = 1;
            ppi[i] = (int16_t)npop;
          }
        ++npop;
        wave_sync();
      }
    }
    if (lane == 0) {
      int keep = npop;
      if (a.cost) {
        // the adaptive budget (CaDDTree's stopping rule, section 2.5, in the pop
        // loop, section 3.4): pop n is kept while theta(n) = (1 + Phi(n)) /
        // (C_d + C_v(n)) improves on theta(n - 1), Phi(n) = sum of exp(g) over
        // the first n pops.  The rule only truncates the pop sequence.
        const float cd = a.cost[0];
        float phi = 0.0f, theta = 1.0f / (cd + a.cost[1]);
        keep = 0;
        for (int i = 0; i < npop; ++i) {
          const float pi = exp_hw(ng[order[i]]);
          const float th = (1.0f + phi + pi) / (cd + a.cost[2 + i]);
          if (!(th > theta)) break;
          phi += pi;
          theta = th;
          keep = i + 1;
        }
      }
      scal[S_NPOP] = keep;
    }
  }
  __syncthreads();

  // ---- emission ---------------------------------------------------------------
  const int npop = scal[S_NPOP];
  const int W32 = (B + 31) / 32;
  for (int i = tid; i < B; i += NT) {
    for (int w = 0; w < W32; ++w) anc[i * 8 + w] = 0;
    if (i < npop) {
      const int node = order[i];
      otok[i] = ntok[node];
      opar[i] = ppi[node];
      odep[i] = ndepth[node];
      opos[i] = a.pos_offset + ndepth[node];
      osc[i] = ng[node];
      // parents pop strictly earlier, so the walk ends within depth <= L steps
      int j = i;
      for (int step = 0; j >= 0 && step <= L; ++step) {
        anc[i * 8 + (j >> 5)] |= 1u << (j & 31);
        const int pj = ppi[order[j]];
        j = pj < j ? pj : -1;
      }
    } else {
      otok[i] = -1;
      opar[i] = -1;
      odep[i] = 0;
      opos[i] = a.pos_offset;
      osc[i] = NEG_INF;
    }
  }
  __syncthreads();
  for (int idx = tid; idx < B * B; idx += NT) {
    const int i = idx / B, j = idx % B;
    omask[idx] = (uint8_t)((anc[i * 8 + (j >> 5)] >> (j & 31)) & 1u);
  }
  if (tid == 0) {
    o.n_nodes[t] = npop;
    o.status[t] = scal[S_STATUS];
  }
  drain();
}

}  // namespace

int expand_group_size(int d_h, int num_cus, int num_xcd, int batch, int M, int L, int nchunks,
                      size_t max_lds) {
  // (a smaller group can need less LDS: fewer units per member than 128 take
  // a 24 KB block for the gates' k-split partial sums; d_h 768 and 1024 fit
  // at 8 members, not at 16)
  int G = 16;
  while (G > 1 && (d_h / G < 32 || (d_h / G) % 16 != 0 ||
                   num_xcd * G * ((batch + num_xcd - 1) / num_xcd) > num_cus ||
                   expand_lds_bytes(d_h, G, M, nchunks, L) > max_lds))
    G >>= 1;
  return G;
}

int expand_group_size(const dt_plan *p, int batch) {
  return expand_group_size(p->d_h, p->num_cus, p->num_xcd, batch, p->M, p->L,
                           scan_geom(batch * p->L, p->V, p->M).nchunks, p->max_lds);
}

size_t expand_lds_bytes(int dh, int G, int M, int nchunks, int L, int rj, int wbytes) {
  return (size_t)lds_layout(dh, G, M, nchunks, L, rj, wbytes).total;
}

size_t expand_part_bytes(const dt_plan *p, int batch) {
  const int G = expand_group_size(p, batch);
  return (size_t)batch * 2 * G * CH * mp_of(p->M) * sizeof(float);
}

hipError_t launch_expand(const dt_plan *p, int batch, const float *h0, float inv_tau,
                         const Workspace &ws, const dt_tree *out, hipStream_t s, hipEvent_t t0,
                         hipEvent_t t1, const ExpMode &mode) {
  ExpArgs a;
  const ScanGeom g = scan_geom(batch * p->L, p->V, p->M);
  a.L = p->L;
  a.M = p->M;
  a.B = mode.B > 0 ? mode.B : p->B;
  a.k = mode.k > 0 ? mode.k : p->k;
  a.nocorr = mode.nocorr;
  a.emit = mode.emit;
  a.skip_merge = mode.skip_merge;
  a.menu_in = mode.menu_in;
  a.menu_out = mode.menu_out;
  a.stats = mode.stats;
  a.cost = (mode.emit && p->frontier_w == 0) ? p->cost : nullptr;
  a.dh = p->d_h;
  a.G = expand_group_size(p, batch);
  a.norm_mode = p->norm_mode;
  a.pos_offset = p->pos_offset;
  a.ecap = ws.ecap;
  a.batch = batch;
  a.nchunks = g.nchunks;
  a.nxcd = p->num_xcd;
  a.W = mode.emit ? p->frontier_w : 0;
  a.spin_limit = p->spin_limit > 0 ? p->spin_limit : kSpinLimit;
  a.use_us = !mode.head && us_fits(p->d_h, a.G, p->M, p->L) &&
             (size_t)p->V * p->d_h * 4 < (size_t)1 << 31;
  a.use_ids = a.use_us || mode.head != nullptr;
  a.rank = a.RJ = a.ld1 = a.d_H = 0;
  a.w1 = a.w2 = nullptr;
  a.ha = nullptr;
  a.hpart = nullptr;
  if (mode.head) {
    a.rank = mode.head->rank;
    a.RJ = mode.head->rank / a.G;
    a.d_H = mode.head->d_H;
    a.ld1 = mode.head->d_H + p->d_h;
    a.w1 = mode.head->w1;
    a.w2 = mode.head->w2;
    a.ha = mode.head->a;
    a.hpart = mode.head->hpart;
  }
  a.inv_tau = inv_tau;
  a.c2 = 1.4426950408889634f * inv_tau;
  a.ckeys = ws.chunk_keys;
  a.ctail = ws.chunk_tail;
  a.cflag = ws.chunk_flag;
  a.cand = ws.cand;
  a.candv = ws.candv;
  a.tailR = ws.tail;
  a.rflag = ws.row_flag;
  a.P_all = p->P_all;
  a.U_all = p->U_all;
  // (the marginals carry no E[v] . b_c term)
  a.c_all = ((mode.nocorr && !mode.menu_in) || mode.head) ? nullptr : p->c_all;
  a.whh = p->whh_t;
  a.b_hh = p->b_hh;
  a.h0 = h0;
  a.states = ws.states;
  a.part = ws.part;
  a.bar = mode.bar ? mode.bar : ws.bar;
  a.out = *out;
  const size_t lds = expand_lds_bytes(p->d_h, a.G, p->M, g.nchunks, p->L, mode.head ? a.RJ : 0,
                                      mode.head ? (p->wdt == DT_BF16 ? 2 : 4) : 0);
  // shapes with a compiled specialisation: Qwen3 drafters (d_h = 512, M = 64,
  // L = 16) with bf16 weights at G = 16 (one to eight trees) and G = 8
  const void *fn;
  const bool arms = mode.nocorr || mode.menu_in || mode.menu_out || !mode.emit || mode.skip_merge;
  const bool qwen = p->wdt == DT_BF16 && a.dh == 512 && a.M == 64 && a.L == 16;
  if (mode.head) {
    if (qwen && a.G == 16)
      fn = (const void *)expand_kernel<uint16_t, 512, 16, 64, 16, false, true>;
    else if (qwen && a.G == 8)
      fn = (const void *)expand_kernel<uint16_t, 512, 8, 64, 16, false, true>;
    else
      fn = p->wdt == DT_BF16 ? (const void *)expand_kernel<uint16_t, 0, 0, 0, 0, false, true>
                             : (const void *)expand_kernel<float, 0, 0, 0, 0, false, true>;
  } else if (arms)
    fn = p->wdt == DT_BF16 ? (const void *)expand_kernel<uint16_t, 0, 0, 0, 0, true>
                           : (const void *)expand_kernel<float, 0, 0, 0, 0, true>;
  else if (p->wdt == DT_BF16 && a.dh == 512 && a.M == 64 && a.L == 16 && a.G == 16)
    fn = (const void *)expand_kernel<uint16_t, 512, 16, 64, 16, false>;
  else if (p->wdt == DT_BF16 && a.dh == 512 && a.M == 64 && a.L == 16 && a.G == 8)
    fn = (const void *)expand_kernel<uint16_t, 512, 8, 64, 16, false>;
  else if (p->wdt == DT_BF16)
    fn = (const void *)expand_kernel<uint16_t, 0, 0, 0, 0, false>;
  else
    fn = (const void *)expand_kernel<float, 0, 0, 0, 0, false>;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  // G > 1: the grid is at most one workgroup per CU (expand_group_size), so
  // every member is resident on an otherwise idle device; members take their
  // slots in start order and every wait is bounded (DT_TREE_TIMEOUT).
  const int grid = a.G > 1 ? a.nxcd * a.G * ((batch + a.nxcd - 1) / a.nxcd) : batch;
  void *args[] = {&a};
  if (t0)
    e = hipExtLaunchKernel(fn, dim3(grid), dim3(NT), args, lds, s, t0, t1, 0);
  else
    e = hipLaunchKernel(fn, dim3(grid), dim3(NT), args, lds, s);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

}  // namespace dt
