// S3-S5: best-first conditional expansion and emission (Alg. 1 steps 2-4;
// section 3.1 conditional children; section 3.5 verification mask).
//
// One workgroup (1024 threads) builds one tree.  The heap of Alg. 1 pops nodes
// in non-increasing score order, and a child never scores above its parent
// (log-probs are <= 0), so the popped set is the top-B of the candidate tree
// (the frontier argument of Appendix B).  A node whose score is below the B-th
// best score already known can therefore never be popped.  The kernel uses this
// in two phases:
//
//  A. Speculative, depth-synchronous expansion.  Starting from the root's
//     children, every known node that is not expanded, is above depth L, and
//     scores at least the current B-th best known score is expanded, a batch of
//     up to 16 nodes at a time: the GRU advances its path state (split-bf16
//     MFMA against the packed W_hh, fp32 accumulation), the correction of the
//     next depth's slice is one fp32 MFMA against the folded U rows, and the
//     top-k children are appended.  This repeats until no node qualifies; every
//     node the heap can pop below depth L is then expanded.
//  B. Exact replay of the heap: B pops by (score desc, insertion order asc),
//     where insertion order is (parent's pop index, child rank) -- the order in
//     which Alg. 1 pushes.  Ties therefore resolve exactly as in the heap.
//
// Emission writes the popped nodes in pop order with parent pop indices,
// depths, position ids, scores and the ancestor-or-self mask.
#include "dt_internal.h"

namespace dt {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int NT = kExpThreads;
constexpr int NW = NT / 64;
constexpr int NC = kNodeCap;
constexpr int CH = kChunkNodes;
static_assert(CH == 16, "MFMA column count");

struct ExpArgs {
  int L, M, B, k, dh, norm_mode, pos_offset, ecap, batch;
  float inv_tau;
  const int32_t *cand;
  const float *candv;
  const float *tail;
  const int32_t *rflag;
  const float *P_all;  // [V][3dh] W_ih E[v] + b_ih
  const float *U_all;  // [V][dh]  W_c^T E[v]
  const float *c_all;  // [V]      E[v] . b_c
  const void *whh;
  const float *b_hh;
  const float *h0;
  float *states;
  dt_tree out;
};

// LDS carve (byte offsets), identical on host and device
struct Lds {
  int ng, ntok, nparent, nstate, nslot, ndepth, nrank, nexp, newidx, elist;
  int ins, popd, ppi, order, anc;
  int Sp, Sn, part, ell, rnk, chunk, scal, total;
};

__host__ __device__ inline Lds lds_layout(int dh, int M) {
  Lds l;
  int o = 0;
  auto take = [&](int bytes) {
    int r = o;
    o += (bytes + 15) / 16 * 16;
    return r;
  };
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
  l.ins = take(NC);
  l.popd = take(NC);
  l.ppi = take(NC * 2);
  l.order = take(kMaxB * 2);
  l.anc = take(kMaxB * 8 * 4);
  l.Sp = take(CH * dh * 4);
  l.Sn = take(CH * dh * 4);
  l.part = take(NW * 16 * CH * 4);
  const int MP = (M + 63) / 64 * 64;
  l.ell = take(CH * MP * 4);
  l.rnk = take(CH * MP * 2);
  l.chunk = take(CH * 2);
  l.scal = take(64 * 4);
  l.total = o;
  return l;
}

// scalar slots in LDS
enum { S_NN, S_VB, S_NEXP, S_STATUS, S_NE, S_NC, S_TOT, S_STOP, S_NPOP, S_CNT0 };

__device__ inline uint16_t f2bf(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ inline float bf2f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

__device__ inline float sigmoidf_(float x) { return 1.0f / (1.0f + expf(-x)); }

__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

__device__ inline uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint64_t p = __shfl_xor(v, o);
    v = p > v ? p : v;
  }
  return v;
}
__device__ inline float wave_max_f(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ inline float wave_sum_f(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ inline float wave_min_f(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o));
  return v;
}

// ordered, exclusive prefix over a predicate evaluated for i = tid + NT*r;
// returns the position of element i among the true ones and the total
struct Compact {
  int pos;
  int total;
};

__device__ inline Compact block_compact(bool pred, int *wcnt /* NW+1 ints in LDS */) {
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
  Compact r;
  r.pos = base + __popcll(b & below);
  r.total = tot;
  return r;
}

template <typename TW>
struct WhhOps;

// bf16 weights: 16x16x32 bf16 MFMA, path state split as hi + mid + lo
template <>
struct WhhOps<uint16_t> {
  static __device__ inline void gates(const ExpArgs &a, const float *Sp, int u, f32x4 (&acc)[3]) {
    const int lane = threadIdx.x & 63;
    const int dh = a.dh, nks = dh / 32;
    const uint4 *W = static_cast<const uint4 *>(a.whh);
    const int c = lane & 15, kq = (lane >> 4) * 8;
#pragma unroll
    for (int g = 0; g < 3; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int ks = 0; ks < nks; ++ks) {
      const float *s = Sp + c * dh + ks * 32 + kq;
      const float4 s0 = *reinterpret_cast<const float4 *>(s);
      const float4 s1 = *reinterpret_cast<const float4 *>(s + 4);
      const float x[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
      bf16x8 hi, mi, lo;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint16_t h = f2bf(x[e]);
        const float r1 = x[e] - bf2f(h);
        const uint16_t m = f2bf(r1);
        const float r2 = r1 - bf2f(m);
        const uint16_t l = f2bf(r2);
        hi[e] = __builtin_bit_cast(__bf16, h);
        mi[e] = __builtin_bit_cast(__bf16, m);
        lo[e] = __builtin_bit_cast(__bf16, l);
      }
#pragma unroll
      for (int g = 0; g < 3; ++g) {
        const uint4 wv = W[((size_t)(u * 3 + g) * nks + ks) * 64 + lane];
        const bf16x8 wa = __builtin_bit_cast(bf16x8, wv);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, lo, acc[g], 0, 0, 0);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, mi, acc[g], 0, 0, 0);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, hi, acc[g], 0, 0, 0);
      }
    }
  }
};

// fp32 weights: 16x16x4 fp32 MFMA, four per k-group of 16
template <>
struct WhhOps<float> {
  static __device__ inline void gates(const ExpArgs &a, const float *Sp, int u, f32x4 (&acc)[3]) {
    const int lane = threadIdx.x & 63;
    const int dh = a.dh, nq = dh / 16;
    const float4 *W = static_cast<const float4 *>(a.whh);
    const int c = lane & 15, kq = (lane >> 4) * 4;
#pragma unroll
    for (int g = 0; g < 3; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int q = 0; q < nq; ++q) {
      const float4 b = *reinterpret_cast<const float4 *>(Sp + c * dh + q * 16 + kq);
#pragma unroll
      for (int g = 0; g < 3; ++g) {
        const float4 wv = W[((size_t)(u * 3 + g) * nq + q) * 64 + lane];
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(wv.x, b.x, acc[g], 0, 0, 0);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(wv.y, b.y, acc[g], 0, 0, 0);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(wv.z, b.z, acc[g], 0, 0, 0);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(wv.w, b.w, acc[g], 0, 0, 0);
      }
    }
  }
};

template <typename TW>
__global__ __launch_bounds__(NT) void expand_kernel(ExpArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const Lds ly = lds_layout(a.dh, a.M);
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
  uint8_t *ins = reinterpret_cast<uint8_t *>(smem + ly.ins);
  uint8_t *popd = reinterpret_cast<uint8_t *>(smem + ly.popd);
  int16_t *ppi = reinterpret_cast<int16_t *>(smem + ly.ppi);
  int16_t *order = reinterpret_cast<int16_t *>(smem + ly.order);
  uint32_t *anc = reinterpret_cast<uint32_t *>(smem + ly.anc);
  float *Sp = reinterpret_cast<float *>(smem + ly.Sp);
  float *Sn = reinterpret_cast<float *>(smem + ly.Sn);
  float *part = reinterpret_cast<float *>(smem + ly.part);
  float *ell = reinterpret_cast<float *>(smem + ly.ell);
  int16_t *rnk = reinterpret_cast<int16_t *>(smem + ly.rnk);
  int16_t *cl = reinterpret_cast<int16_t *>(smem + ly.chunk);
  int *scal = reinterpret_cast<int *>(smem + ly.scal);
  float *scalf = reinterpret_cast<float *>(smem + ly.scal);
  int *wcnt = scal + 32;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t = blockIdx.x;
  const int L = a.L, M = a.M, B = a.B, dh = a.dh;
  const int MP = (M + 63) / 64 * 64;
  const float NEG_INF = -__builtin_huge_valf();
  // nodes per chunk, so that one chunk's children (<= k each) fit the table
  int chunk_cap = (NC - B - 64) / a.k;
  chunk_cap = chunk_cap > CH ? CH : (chunk_cap < 1 ? 1 : chunk_cap);

  dt_tree o = a.out;
  int32_t *otok = o.tokens + (size_t)t * B;
  int32_t *opar = o.parents + (size_t)t * B;
  int32_t *odep = o.depth + (size_t)t * B;
  int32_t *opos = o.position_ids + (size_t)t * B;
  float *osc = o.scores + (size_t)t * B;
  uint8_t *omask = o.mask + (size_t)t * B * B;

  // ---- per-tree data errors -------------------------------------------------
  if (tid == 0) {
    int f = 0;
    for (int d = 0; d < L; ++d) f |= a.rflag[t * L + d];
    scal[S_STATUS] = f;
    scal[S_NN] = 0;
    scalf[S_VB] = NEG_INF;
    scal[S_NEXP] = 0;
    scal[S_STOP] = 0;
  }
  __syncthreads();
  if (scal[S_STATUS] & DT_TREE_NONFINITE) {
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
    return;
  }

  // ---- expand one chunk of nodes (all at depth d; d = 0 is the root) -------
  auto expand_chunk = [&](const int16_t *cn, int nc, int d) {
    // 1. path states of the parents (root: h0)
    for (int idx = tid; idx < CH * dh; idx += NT) {
      const int c = idx / dh, j = idx % dh;
      float v = 0.0f;
      if (c < nc) {
        const int par = (d == 0) ? -1 : nparent[cn[c]];
        if (par < 0)
          v = a.h0 ? a.h0[(size_t)t * dh + j] : 0.0f;
        else
          v = a.states[((size_t)t * a.ecap + nstate[par]) * dh + j];
      }
      Sp[idx] = v;
    }
    if (d > 0 && tid < nc) nstate[cn[tid]] = (int16_t)(scal[S_NEXP] + tid);
    __syncthreads();
    // 2. GRU along each node's own path (Domino's causal encoder); each wave
    //    owns whole groups of 16 hidden units, so it can finish a group alone
    const float *Scur = Sp;  // state the children are scored from
    if (d > 0) {
      const int ngr = dh / 16;
      const int c = lane & 15;
      const int node = c < nc ? cn[c] : 0;
      const float *prow = a.P_all + (size_t)(c < nc ? ntok[node] : 0) * (3 * dh);
      float *srow = a.states + ((size_t)t * a.ecap + (c < nc ? nstate[node] : 0)) * dh;
      for (int u = wave; u < ngr; u += NW) {
        f32x4 gh[3];
        WhhOps<TW>::gates(a, Sp, u, gh);
        if (c < nc) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int j = 16 * u + (lane >> 4) * 4 + i;
            const float hr = gh[0][i] + a.b_hh[j];
            const float hz = gh[1][i] + a.b_hh[dh + j];
            const float hn = gh[2][i] + a.b_hh[2 * dh + j];
            const float r = sigmoidf_(prow[j] + hr);
            const float z = sigmoidf_(prow[dh + j] + hz);
            const float n = tanhf(prow[2 * dh + j] + r * hn);
            const float sv = (1.0f - z) * n + z * Sp[c * dh + j];
            Sn[c * dh + j] = sv;
            srow[j] = sv;
          }
        }
      }
      __syncthreads();
      Scur = Sn;
    }
    if (d >= L) return;
    // 3. correction of depth d+1's slice: delta[m][c] = U[m] . S_c (fp32 MFMA)
    const int RT = (M + 15) / 16;
    const int F = NW / RT;
    const int nq = dh / 16;
    const size_t rbase = (size_t)(t * L + d) * M;  // depth d+1 rows
    if (wave < RT * F) {
      const int rt = wave % RT, f = wave / RT;
      const int q0 = (nq * f) / F, q1 = (nq * (f + 1)) / F;
      const int m = rt * 16 + (lane & 15);
      const int c = lane & 15, kq = (lane >> 4) * 4;
      const float *urow = a.U_all + (size_t)(m < M ? a.cand[rbase + m] : 0) * dh;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int q = q0; q < q1; ++q) {
        float4 av = make_float4(0.f, 0.f, 0.f, 0.f);
        if (m < M) av = *reinterpret_cast<const float4 *>(urow + q * 16 + kq);
        const float4 bv = *reinterpret_cast<const float4 *>(Scur + c * dh + q * 16 + kq);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.x, bv.x, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.y, bv.y, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.z, bv.z, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.w, bv.w, acc, 0, 0, 0);
      }
      // lane l, register i: slot rt*16 + (l/16)*4 + i, node l%16
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int slot = rt * 16 + (lane >> 4) * 4 + i;
        part[(f * RT * 16 + slot) * CH + c] = acc[i];
      }
    }
    __syncthreads();
    // 4. children of node `wave`: normalise, rank, keep the top-k above vB
    const float vB = scalf[S_VB];
    const float R = a.tail[t * L + d];
    int kc = 0;
    if (wave < nc) {
      const int c = wave;
      const float gpar = (d == 0) ? 0.0f : ng[cn[c]];
      float zv[4];
      float mx = NEG_INF;
      for (int s = 0; s < MP / 64; ++s) {
        const int m = lane + 64 * s;
        float z = NEG_INF;
        if (m < M) {
          const float x = a.candv[rbase + m];
          if (x > NEG_INF) {
            float dl = a.c_all[a.cand[rbase + m]];
            for (int f = 0; f < F; ++f) dl += part[(f * RT * 16 + m) * CH + c];
            z = (x + dl) * a.inv_tau;
          }
        }
        zv[s] = z;
        mx = fmaxf(mx, z);
      }
      mx = wave_max_f(mx);
      const bool tail = (a.norm_mode == DT_NORM_TAIL) && R > NEG_INF;
      if (tail) mx = fmaxf(mx, R);
      float sum = 0.0f;
      for (int s = 0; s < MP / 64; ++s) sum += (zv[s] > NEG_INF) ? expf(zv[s] - mx) : 0.0f;
      sum = wave_sum_f(sum);
      if (tail) sum += expf(R - mx);
      const float logZ = mx + logf(sum);
      for (int s = 0; s < MP / 64; ++s) {
        const int m = lane + 64 * s;
        ell[c * MP + m] = (zv[s] > NEG_INF) ? zv[s] - logZ : NEG_INF;
      }
      wave_sync();
      // rank of each live slot by (ell desc, slot asc); keep ranks < k with g >= vB
      for (int s = 0; s < MP / 64; ++s) {
        const int m = lane + 64 * s;
        const float lm = ell[c * MP + m];
        int rank = 0;
        if (lm > NEG_INF) {
          for (int m2 = 0; m2 < M; ++m2) {
            const float l2 = ell[c * MP + m2];
            rank += (l2 > lm) || (l2 == lm && m2 < m);
          }
        }
        const bool keep = lm > NEG_INF && rank < a.k && gpar + lm >= vB;
        kc += __popcll(__ballot(keep));
        rnk[c * MP + m] = keep ? (int16_t)rank : (int16_t)-1;
      }
      if (lane == 0) wcnt[c] = kc;
    } else if (wave < CH && lane == 0) {
      wcnt[wave] = 0;
    }
    __syncthreads();
    // 5. append children (node order, then rank order) to the node table
    int base = scal[S_NN];
    int tot = 0;
    for (int c = 0; c < CH; ++c) tot += (c < nc) ? wcnt[c] : 0;
    if (wave < nc) {
      const int c = wave;
      int off = base;
      for (int c2 = 0; c2 < c; ++c2) off += wcnt[c2];
      const float gpar = (d == 0) ? 0.0f : ng[cn[c]];
      for (int s = 0; s < MP / 64; ++s) {
        const int m = lane + 64 * s;
        const int rk = rnk[c * MP + m];
        if (m < M && rk >= 0) {
          const int pos = off + rk;
          if (pos < NC) {
            ng[pos] = gpar + ell[c * MP + m];
            ntok[pos] = a.cand[rbase + m];
            nslot[pos] = (int16_t)m;
            ndepth[pos] = (uint8_t)(d + 1);
            nparent[pos] = (d == 0) ? (int16_t)-1 : cn[c];
            nrank[pos] = (uint8_t)rk;
            nstate[pos] = -1;
            nexp[pos] = 0;
          }
        }
      }
    }
    __syncthreads();
    if (tid == 0) {
      int nn = base + tot;
      if (nn > NC) {
        nn = NC;
        scal[S_STATUS] |= DT_TREE_TRUNCATED;  // table overflow (massive exact ties)
      }
      scal[S_NN] = nn;
      if (d > 0) scal[S_NEXP] += nc;
    }
    if (d > 0 && tid < nc) nexp[cn[tid]] = 1;
    __syncthreads();
  };

  // ---- vB = B-th best known score; drop nodes below it when room is needed --
  auto update_vb = [&](bool compact) {
    const int nn = scal[S_NN];
    if (nn >= B) {
      float best = __builtin_huge_valf();
      for (int i = tid; i < nn; i += NT) {
        const float gi = ng[i];
        int cnt = 0;
        for (int j = 0; j < nn; ++j) cnt += ng[j] > gi;
        if (cnt < B) best = fminf(best, gi);
      }
      best = wave_min_f(best);
      if (lane == 0) scalf[S_CNT0 + wave] = best;
      __syncthreads();
      if (tid == 0) {
        float v = scalf[S_CNT0];
        for (int w = 1; w < NW; ++w) v = fminf(v, scalf[S_CNT0 + w]);
        scalf[S_VB] = v;
      }
      __syncthreads();
    }
    if (!compact || nn < B) return;
    const float vB = scalf[S_VB];
    // keep g >= vB (parents always score at least their children, so links stay valid)
    for (int r0 = 0; r0 < nn; r0 += NT) {
      const int i = r0 + tid;
      const bool keep = i < nn && ng[i] >= vB;
      Compact cp = block_compact(keep, wcnt);
      if (i < nn) newidx[i] = keep ? (int16_t)(cp.pos + (r0 ? scal[S_TOT] : 0)) : (int16_t)-1;
      __syncthreads();
      if (tid == 0) scal[S_TOT] = (r0 ? scal[S_TOT] : 0) + cp.total;
      __syncthreads();
    }
    const int kept = scal[S_TOT];
    // move (each thread owns at most two entries; read all, then write)
    float rg[2];
    int rt[2], rp[2], rs[2], rsl[2], rd[2], rr[2], re[2], dst[2];
    for (int q = 0; q < 2; ++q) {
      const int i = tid + q * NT;
      dst[q] = (i < nn) ? newidx[i] : -1;
      if (dst[q] >= 0) {
        rg[q] = ng[i];
        rt[q] = ntok[i];
        rp[q] = nparent[i] >= 0 ? newidx[nparent[i]] : -1;
        rs[q] = nstate[i];
        rsl[q] = nslot[i];
        rd[q] = ndepth[i];
        rr[q] = nrank[i];
        re[q] = nexp[i];
      }
    }
    __syncthreads();
    for (int q = 0; q < 2; ++q) {
      if (dst[q] >= 0) {
        const int j = dst[q];
        ng[j] = rg[q];
        ntok[j] = rt[q];
        nparent[j] = (int16_t)rp[q];
        nstate[j] = (int16_t)rs[q];
        nslot[j] = (int16_t)rsl[q];
        ndepth[j] = (uint8_t)rd[q];
        nrank[j] = (uint8_t)rr[q];
        nexp[j] = (uint8_t)re[q];
      }
    }
    __syncthreads();
    if (tid == 0) scal[S_NN] = kept;
    __syncthreads();
  };

  // ---- phase A ---------------------------------------------------------------
  expand_chunk(nullptr, 1, 0);  // root: children at depth 1 scored from h0
  update_vb(false);
  for (int iter = 0; iter < L; ++iter) {
    // eligible: known, unexpanded, above depth L, score >= vB (index order)
    const int nn = scal[S_NN];
    const float vB = scalf[S_VB];
    for (int r0 = 0; r0 < nn; r0 += NT) {
      const int i = r0 + tid;
      const bool e = i < nn && !nexp[i] && ndepth[i] < L && ng[i] >= vB;
      Compact cp = block_compact(e, wcnt);
      const int off = r0 ? scal[S_NE] : 0;
      if (e) elist[off + cp.pos] = (int16_t)i;
      __syncthreads();
      if (tid == 0) scal[S_NE] = off + cp.total;
      __syncthreads();
    }
    const int ne = nn ? scal[S_NE] : 0;
    if (ne == 0) break;
    int pos = 0;
    while (pos < ne) {
      __syncthreads();  // everyone has read the previous chunk's scalars
      // next chunk: up to chunk_cap nodes that still score >= vB
      if (tid == 0) {
        const float v = scalf[S_VB];
        int c = 0;
        int p = pos;
        while (p < ne && c < chunk_cap) {
          const int i = elist[p++];
          if (i >= 0 && ng[i] >= v) cl[c++] = (int16_t)i;
        }
        scal[S_NC] = c;
        scal[S_TOT] = p;
        if (c && scal[S_NEXP] + c > a.ecap) {
          scal[S_STATUS] |= DT_TREE_TRUNCATED;
          scal[S_STOP] = 1;
        }
      }
      __syncthreads();
      const int nc = scal[S_NC];
      pos = scal[S_TOT];
      if (scal[S_STOP]) break;
      if (nc == 0) continue;
      // make room for the children of this chunk
      const bool need = scal[S_NN] + nc * a.k > NC - CH;
      if (need) {
        update_vb(true);
        // remap the rest of the eligible list and the chunk
        for (int p = tid; p < ne; p += NT) {
          const int i = elist[p];
          elist[p] = (i >= 0) ? newidx[i] : (int16_t)-1;
        }
        __syncthreads();
        if (tid == 0) {
          int c2 = 0;
          for (int c = 0; c < nc; ++c) {
            const int i = newidx[cl[c]];
            if (i >= 0) cl[c2++] = (int16_t)i;
          }
          scal[S_NC] = c2;
        }
        __syncthreads();
      }
      const int nc2 = scal[S_NC];
      if (nc2 == 0) continue;
      expand_chunk(cl, nc2, ndepth[cl[0]]);
      update_vb(false);
    }
    if (scal[S_STOP]) break;
  }

  // ---- phase B: exact replay of the heap --------------------------------------
  const int nn = scal[S_NN];
  if (wave == 0) {
    for (int i = lane; i < nn; i += 64) {
      ins[i] = nparent[i] < 0;
      popd[i] = 0;
      ppi[i] = -1;
    }
    wave_sync();
    int npop = 0;
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
    if (lane == 0) scal[S_NPOP] = npop;
  }
  __syncthreads();

  // ---- emission -----------------------------------------------------------------
  const int npop = scal[S_NPOP];
  const int W32 = (B + 31) / 32;
  for (int i = tid; i < B; i += NT) {
    if (i < npop) {
      const int node = order[i];
      otok[i] = ntok[node];
      opar[i] = ppi[node];
      odep[i] = ndepth[node];
      opos[i] = a.pos_offset + ndepth[node];
      osc[i] = ng[node];
      for (int w = 0; w < W32; ++w) anc[i * 8 + w] = 0;
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
      for (int w = 0; w < W32; ++w) anc[i * 8 + w] = 0;
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
}

}  // namespace

size_t expand_lds_bytes(int dh, int M) { return (size_t)lds_layout(dh, M).total; }

hipError_t launch_expand(const dt_plan *p, int batch, const float *h0, float inv_tau,
                         const Workspace &ws, const dt_tree *out, hipStream_t s) {
  ExpArgs a;
  a.L = p->L;
  a.M = p->M;
  a.B = p->B;
  a.k = p->k;
  a.dh = p->d_h;
  a.norm_mode = p->norm_mode;
  a.pos_offset = p->pos_offset;
  a.ecap = ws.ecap;
  a.batch = batch;
  a.inv_tau = inv_tau;
  a.cand = ws.cand;
  a.candv = ws.candv;
  a.tail = ws.tail;
  a.rflag = ws.row_flag;
  a.P_all = p->P_all;
  a.U_all = p->U_all;
  a.c_all = p->c_all;
  a.whh = p->whh_t;
  a.b_hh = p->b_hh;
  a.h0 = h0;
  a.states = ws.states;
  a.out = *out;
  const size_t lds = expand_lds_bytes(p->d_h, p->M);
  if (p->wdt == DT_BF16) {
    hipFuncSetAttribute((const void *)expand_kernel<uint16_t>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(expand_kernel<uint16_t>, dim3(batch), dim3(NT), lds, s, a);
  } else {
    hipFuncSetAttribute((const void *)expand_kernel<float>,
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(expand_kernel<float>, dim3(batch), dim3(NT), lds, s, a);
  }
  return hipGetLastError();
}

}  // namespace dt
