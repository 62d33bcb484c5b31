// Domino's own correction head on the tree builder (section 2.3): the
// correction of slot m of depth d's slice, for a node with path state S, is
//   delta_m = W_2[cand_d[m]] . SiLU(W_1 [H_d; S])
// with a rank-r bottleneck and no biases, in place of the linear head's
// E[v] . (W_c S + b_c).  Scoring, normalisation, ties and emission are the
// same as the default path's (Alg. 1; section 3.2 for the slice).
//
// This file holds the tree kernel for shapes the expansion kernel does not
// take: one workgroup per tree, the exact row merge, then the best-first heap
// of Alg. 1 in LDS, one pop at a time.  a[row][r] = W_1^H H_row, the half of
// W_1 [H_d; S] that does not depend on the path, comes from the scan launch.
// A pop advances the popped node's GRU state from its parent's state and
// W_hh S_parent (kept per popped node, computed the first time one of its
// children is popped), forms y = SiLU(a_d + W_1^S S) and the slice's
// corrections W_2[cand] . y, and pushes its top-k children in rank order
// (one wave's bitonic sort of the slice).
#include "dt_internal.h"
#include "dt_select.h"
#include <hip/hip_ext.h>

namespace dt {
namespace {

constexpr int kHT = 512;        // threads of the tree kernel

__device__ inline void load8(const float *p, float (&v)[8]) {
  const float4 a = *reinterpret_cast<const float4 *>(p);
  const float4 b = *reinterpret_cast<const float4 *>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ inline void load8(const uint16_t *p, float (&v)[8]) {
  const uint4 q = *reinterpret_cast<const uint4 *>(p);
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}

// w[0..7] . x[0..7] with x 16-byte aligned (LDS)
__device__ inline float dot8(const float (&w)[8], const float *x) {
  const float4 a = *reinterpret_cast<const float4 *>(x);
  const float4 b = *reinterpret_cast<const float4 *>(x + 4);
  float s = w[0] * a.x;
  s = fmaf(w[1], a.y, s);
  s = fmaf(w[2], a.z, s);
  s = fmaf(w[3], a.w, s);
  s = fmaf(w[4], b.x, s);
  s = fmaf(w[5], b.y, s);
  s = fmaf(w[6], b.z, s);
  return fmaf(w[7], b.w, s);
}
// sum over the 8 lanes of an aligned group
__device__ inline float sum8(float v) {
  v += __shfl_xor(v, 1);
  v += __shfl_xor(v, 2);
  v += __shfl_xor(v, 4);
  return v;
}
__device__ inline uint64_t wave_max_key(uint64_t v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)v, o), hi = __shfl_xor((uint32_t)(v >> 32), o);
    const uint64_t u = ((uint64_t)hi << 32) | lo;
    v = u > v ? u : v;
  }
  return v;
}

// out[r] = sum_{c < n} W[r * ld + c] x[c] for r < nrows: eight lanes per row,
// eight consecutive columns per lane and chunk (n % 8 == 0; W rows 16-byte
// aligned); x in LDS.  Each pass takes kRU rows and kCU chunks per lane with
// every load issued before the first is used (out-of-range ones read a valid
// address and count zero), so a pass costs one memory round trip.  Every
// thread of the block calls it.
constexpr int kRU = 2, kCU = 4;
template <typename T>
__device__ void rows_dot(const T *W, size_t ld, int nrows, int n, const float *x, float *out) {
  const int grp = threadIdx.x >> 3, sub = threadIdx.x & 7;
  for (int r0 = grp * kRU; r0 < nrows; r0 += (kHT / 8) * kRU) {
    float acc[kRU];
#pragma unroll
    for (int i = 0; i < kRU; ++i) acc[i] = 0.0f;
    for (int c0 = sub * 8; c0 < n; c0 += 64 * kCU) {
      float w[kRU][kCU][8];
#pragma unroll
      for (int i = 0; i < kRU; ++i)
#pragma unroll
        for (int j = 0; j < kCU; ++j) {
          const int r = r0 + i < nrows ? r0 + i : nrows - 1;
          const int c = c0 + 64 * j < n ? c0 + 64 * j : 0;
          load8(W + (size_t)r * ld + c, w[i][j]);
        }
#pragma unroll
      for (int i = 0; i < kRU; ++i)
#pragma unroll
        for (int j = 0; j < kCU; ++j) {
          const int c = c0 + 64 * j;
          const float v = dot8(w[i][j], x + (c < n ? c : 0));
          acc[i] += c < n ? v : 0.0f;
        }
    }
#pragma unroll
    for (int i = 0; i < kRU; ++i) {
      const float v = sum8(acc[i]);
      if (sub == 0 && r0 + i < nrows) out[r0 + i] = v;
    }
  }
}

struct HeadArgs {
  const uint64_t *ckeys;  // scan segment lists [rows][nchunks][M]
  const float2 *ctail;    // [rows][nchunks]
  const int32_t *cflag;   // [rows][nchunks]
  int nchunks;
  const float *P_all;     // [V][3dh] W_ih E[v] + b_ih + (b_hh on gates r, z)
  const void *whh;        // [3dh][dh] W_hh (weights dtype)
  const float *b_hh;      // [3dh] fp32 (b_hn used)
  const void *w1;         // [rank][d_H + dh]
  const void *w2;         // [V][rank]
  const float *a;         // [rows][rank] W_1^H H
  const float *h0;        // [batch][dh] or null
  float *states;          // [batch][B + 1][dh]: slot 0 the root, slot i + 1 pop i
  float *ghs;             // [batch][B + 1][3dh]: W_hh S of the same slots
  int L, M, B, k, dh, d_H, rank, norm_mode, pos_offset;
  float c2, inv_tau;      // c2 = log2(e) / tau
  const float *cost;      // adaptive budget: C_d, C_v(0..B) (device), or null (fixed budget)
  dt_tree out;
};

// LDS carve of head_tree_kernel (byte offsets); host and device agree
struct HeadLds {
  int key, tok, par, slot, dep, rc, rv, rt, rf, ptok, pg, pdep, ppar, pgh, Sp, Sc, gh, u, y, dl,
      red, scal, total;
};
__host__ __device__ inline int take(int &p, int bytes) {
  const int q = p;
  p += (bytes + 15) & ~15;
  return q;
}
__host__ __device__ inline HeadLds head_lds(int L, int B, int dh, int rank) {
  HeadLds o;
  int p = 0;
  o.key = take(p, 8 * kHeadCap);
  o.tok = take(p, 4 * kHeadCap);
  o.par = take(p, 2 * kHeadCap);
  o.slot = take(p, kHeadCap);
  o.dep = take(p, kHeadCap);
  o.rc = take(p, 4 * 64 * L);
  o.rv = take(p, 4 * 64 * L);
  o.rt = take(p, 4 * L);
  o.rf = take(p, 4 * L);
  o.ptok = take(p, 4 * B);
  o.pg = take(p, 4 * B);
  o.pdep = take(p, 4 * B);
  o.ppar = take(p, 4 * B);
  o.pgh = take(p, 4 * (B + 1));
  o.Sp = take(p, 4 * dh);
  o.Sc = take(p, 4 * dh);
  o.gh = take(p, 12 * dh);
  o.u = take(p, 4 * rank);
  o.y = take(p, 4 * rank);
  o.dl = take(p, 4 * 64);
  o.red = take(p, 8 * (kHT / 64));
  o.scal = take(p, 4 * 8);
  o.total = p;
  return o;
}
enum { H_NE, H_NPOP, H_STATUS };

__device__ inline float sigm(float x) { return 1.0f / (1.0f + expf(-x)); }

template <typename T>
__global__ __launch_bounds__(kHT) void head_tree_kernel(HeadArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int L = a.L, M = a.M, B = a.B, dh = a.dh, R = a.rank;
  const HeadLds ly = head_lds(L, B, dh, R);
  uint64_t *hkey = reinterpret_cast<uint64_t *>(smem + ly.key);
  int32_t *htok = reinterpret_cast<int32_t *>(smem + ly.tok);
  int16_t *hpar = reinterpret_cast<int16_t *>(smem + ly.par);
  uint8_t *hslot = reinterpret_cast<uint8_t *>(smem + ly.slot);
  uint8_t *hdep = reinterpret_cast<uint8_t *>(smem + ly.dep);
  int32_t *rc = reinterpret_cast<int32_t *>(smem + ly.rc);
  float *rv = reinterpret_cast<float *>(smem + ly.rv);
  float *rt = reinterpret_cast<float *>(smem + ly.rt);
  int32_t *rf = reinterpret_cast<int32_t *>(smem + ly.rf);
  int32_t *ptok = reinterpret_cast<int32_t *>(smem + ly.ptok);
  float *pg = reinterpret_cast<float *>(smem + ly.pg);
  int32_t *pdep = reinterpret_cast<int32_t *>(smem + ly.pdep);
  int32_t *ppar = reinterpret_cast<int32_t *>(smem + ly.ppar);
  int32_t *pgh = reinterpret_cast<int32_t *>(smem + ly.pgh);
  float *Sp = reinterpret_cast<float *>(smem + ly.Sp);
  float *Sc = reinterpret_cast<float *>(smem + ly.Sc);
  float *gh = reinterpret_cast<float *>(smem + ly.gh);
  float *uu = reinterpret_cast<float *>(smem + ly.u);
  float *yy = reinterpret_cast<float *>(smem + ly.y);
  float *dl = reinterpret_cast<float *>(smem + ly.dl);
  uint64_t *red = reinterpret_cast<uint64_t *>(smem + ly.red);
  int *scal = reinterpret_cast<int *>(smem + ly.scal);

  const int t = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float NEG_INF = -__builtin_huge_valf();
  const T *whh = static_cast<const T *>(a.whh);
  const T *w1 = static_cast<const T *>(a.w1);
  const T *w2 = static_cast<const T *>(a.w2);
  const size_t ld1 = (size_t)a.d_H + dh;
  float *st = a.states + (size_t)t * (B + 1) * dh;
  float *ghg = a.ghs + (size_t)t * (B + 1) * 3 * dh;

  // ---- Alg. 1 step 1: this tree's rows, one wave per row ---------------------
  for (int d = wave; d < L; d += kHT / 64) {
    const size_t row = (size_t)t * L + d;
    sel::merge_row_wave<false, true>(a.ckeys + row * a.nchunks * M, a.nchunks, M,
                               a.ctail + row * a.nchunks, a.cflag + row * a.nchunks, a.c2,
                               a.inv_tau, rc + 64 * d, rv + 64 * d, rt + d, rf + d, nullptr);
  }
  for (int u = tid; u < dh; u += kHT) {
    const float v = a.h0 ? a.h0[(size_t)t * dh + u] : 0.0f;
    Sc[u] = v;
    st[u] = v;
  }
  for (int i = tid; i <= B; i += kHT) pgh[i] = 0;
  if (tid == 0) {
    scal[H_NE] = 0;
    scal[H_NPOP] = 0;
    scal[H_STATUS] = 0;
  }
  __syncthreads();
  int bad = 0;
  for (int d = 0; d < L; ++d) bad |= rf[d];

  dt_tree o = a.out;
  int32_t *otok = o.tokens + (size_t)t * B;
  int32_t *opar = o.parents + (size_t)t * B;
  int32_t *odep = o.depth + (size_t)t * B;
  int32_t *opos = o.position_ids + (size_t)t * B;
  float *osc = o.scores + (size_t)t * B;
  uint8_t *omask = o.mask + (size_t)t * B * B;

  if (!bad) {
    // children of a node (pop index pi, -1 = the root) at depth d whose state
    // is in Sc: score row d, push the top k (Alg. 1 steps 2-3)
    auto children = [&](int pi, int d, float g) {
      rows_dot(w1 + a.d_H, ld1, R, dh, Sc, uu);  // W_1^S S
      __syncthreads();
      const float *ad = a.a + ((size_t)t * L + d) * R;
      for (int r = tid; r < R; r += kHT) {
        const float v = uu[r] + ad[r];
        yy[r] = v * sigm(v);  // SiLU
      }
      __syncthreads();
      {
        // delta_m = W_2[cand_d[m]] . y, eight lanes per slot
        const int m = tid >> 3, sub = tid & 7;
        if (m < M) {
          const int v = rc[64 * d + m];
          const T *wr = w2 + (size_t)(v >= 0 ? v : 0) * R;
          float acc = 0.0f;
          for (int c0 = sub * 8; c0 < R; c0 += 64 * kCU) {
            float w[kCU][8];
#pragma unroll
            for (int j = 0; j < kCU; ++j) load8(wr + (c0 + 64 * j < R ? c0 + 64 * j : 0), w[j]);
#pragma unroll
            for (int j = 0; j < kCU; ++j) {
              const int c = c0 + 64 * j;
              const float p = dot8(w[j], yy + (c < R ? c : 0));
              acc += c < R ? p : 0.0f;
            }
          }
          acc = sum8(acc);
          if (v < 0) acc = 0.0f;
          if (sub == 0) dl[m] = acc;
        }
      }
      __syncthreads();
      if (wave == 0) {
        const float x = lane < M ? rv[64 * d + lane] : NEG_INF;
        const bool live = x > NEG_INF;
        const float z = live ? (x + dl[lane]) * a.inv_tau : NEG_INF;
        float mx = sel::wave_reduce(z, [](float p, float q) { return fmaxf(p, q); });
        const float Rd = rt[d];
        const bool tail = a.norm_mode == DT_NORM_TAIL && Rd > NEG_INF;
        if (tail) mx = fmaxf(mx, Rd);
        float s = sel::wave_reduce(live ? expf(z - mx) : 0.0f, [](float p, float q) { return p + q; });
        if (tail) s += expf(Rd - mx);
        const float logZ = mx + logf(s);
        const float ell = live ? z - logZ : NEG_INF;
        // rank by (ell desc, slot asc): lane j of the sorted keys holds rank j
        const uint64_t srt = sel::wave_sort64(live ? make_key(ell, (uint32_t)lane) : 0ull, true);
        const int ne = scal[H_NE];
        const bool keep = srt != 0ull && lane < a.k && ne + lane < kHeadCap;
        if (keep) {
          const int e = ne + lane;  // insertion order = rank order
          const int m = (int)key_index(srt);
          hkey[e] = make_key(g + key_value(srt), (uint32_t)e);
          htok[e] = rc[64 * d + m];
          hslot[e] = (uint8_t)m;
          hpar[e] = (int16_t)pi;
          hdep[e] = (uint8_t)(d + 1);
        }
        const int nk = __popcll(__ballot(keep));
        const int nwant = __popcll(__ballot(srt != 0ull && lane < a.k));
        if (lane == 0) {
          scal[H_NE] = ne + nk;
          if (nwant > nk) scal[H_STATUS] |= DT_TREE_TRUNCATED;  // heap full (not reached in range)
        }
      }
      __syncthreads();
    };

    children(-1, 0, 0.0f);
    // adaptive budget (CaDDTree's stopping rule, section 2.5, in the pop loop,
    // section 3.4): Phi and theta of the nodes popped so far (every thread
    // holds the same values)
    float phi = 0.0f, theta = a.cost ? 1.0f / (a.cost[0] + a.cost[1]) : 0.0f;
    for (;;) {
      // pop the best entry: (g desc, insertion asc) is key desc
      const int ne = scal[H_NE];
      uint64_t best = 0ull;
      for (int i = tid; i < ne; i += kHT) best = hkey[i] > best ? hkey[i] : best;
      best = wave_max_key(best);
      if (lane == 0) red[wave] = best;
      __syncthreads();
      best = red[0];
#pragma unroll
      for (int w = 1; w < kHT / 64; ++w) best = red[w] > best ? red[w] : best;
      const int npop = scal[H_NPOP];
      __syncthreads();
      if (best == 0ull || npop >= B) break;
      const int e = (int)key_index(best);
      const float g = key_value(best);
      if (a.cost) {
        // theta(n) with this entry as node n; stop (not kept) when it does not improve
        const float pi = __builtin_amdgcn_exp2f(1.44269504088896341f * g);
        const float th = (1.0f + phi + pi) / (a.cost[0] + a.cost[2 + npop]);
        if (!(th > theta)) break;
        phi += pi;
        theta = th;
      }
      const int tok = htok[e], dep = hdep[e], par = hpar[e];
      if (tid == 0) {
        hkey[e] = 0ull;
        ptok[npop] = tok;
        pg[npop] = g;
        pdep[npop] = dep;
        ppar[npop] = par;
        scal[H_NPOP] = npop + 1;
      }
      if (dep < L) {
        // the popped node's state: GRU(parent state, its token), section 2.3
        const int ps = par + 1;
        for (int u = tid; u < dh; u += kHT) Sp[u] = st[(size_t)ps * dh + u];
        const int have = pgh[ps];
        __syncthreads();
        if (!have) {
          rows_dot(whh, (size_t)dh, 3 * dh, dh, Sp, gh);
          __syncthreads();
          for (int j = tid; j < 3 * dh; j += kHT) ghg[(size_t)ps * 3 * dh + j] = gh[j];
          if (tid == 0) pgh[ps] = 1;
        } else {
          for (int j = tid; j < 3 * dh; j += kHT) gh[j] = ghg[(size_t)ps * 3 * dh + j];
        }
        __syncthreads();
        const float *Pr = a.P_all + (size_t)tok * 3 * dh;
        for (int u = tid; u < dh; u += kHT) {
          const float r = sigm(Pr[u] + gh[u]);
          const float z = sigm(Pr[dh + u] + gh[dh + u]);
          const float n = tanhf(Pr[2 * dh + u] + r * (gh[2 * dh + u] + a.b_hh[2 * dh + u]));
          const float h = (1.0f - z) * n + z * Sp[u];
          Sc[u] = h;
          st[(size_t)(npop + 1) * dh + u] = h;
        }
        __syncthreads();
        children(npop, dep, g);
      }
      __syncthreads();
    }
  }

  // ---- emission in pop order (section 3.5) -------------------------------------
  const int npop = bad ? 0 : scal[H_NPOP];
  for (int i = tid; i < B; i += kHT) {
    const bool in = i < npop;
    otok[i] = in ? ptok[i] : -1;
    opar[i] = in ? ppar[i] : -1;
    odep[i] = in ? pdep[i] : 0;
    opos[i] = a.pos_offset + (in ? pdep[i] : 0);
    osc[i] = in ? pg[i] : NEG_INF;
    uint8_t *row = omask + (size_t)i * B;
    for (int j = 0; j < B; ++j) row[j] = 0;
    if (in)
      for (int p = i; p >= 0; p = ppar[p]) row[p] = 1;
  }
  if (tid == 0) {
    o.n_nodes[t] = npop;
    o.status[t] = bad ? DT_TREE_NONFINITE : scal[H_STATUS];
  }
}

}  // namespace

size_t head_lds_bytes(int L, int B, int dh, int rank) { return (size_t)head_lds(L, B, dh, rank).total; }

HeadWorkspace carve_head(const dt_plan *p, int batch, int rank, char *base) {
  HeadWorkspace hw;
  const ScanGeom g = scan_geom(batch * p->L, p->V, p->M);
  size_t o = carve_scan(base, g, &hw.scan);
  hw.a = reinterpret_cast<float *>(base + o);
  o += align_up((size_t)batch * p->L * rank * sizeof(float), 256);
  hw.states = reinterpret_cast<float *>(base + o);
  o += align_up((size_t)batch * (p->B + 1) * p->d_h * sizeof(float), 256);
  hw.ghs = reinterpret_cast<float *>(base + o);
  o += align_up((size_t)batch * (p->B + 1) * 3 * p->d_h * sizeof(float), 256);
  hw.bytes = o;
  return hw;
}

template <typename T>
static hipError_t launch_head_t(const dt_plan *p, int batch, const void *H, const dt_domino_head &hd,
                                const float *h0, float inv_tau, const HeadWorkspace &hw, dt_tree *out,
                                hipStream_t s, hipEvent_t t0, hipEvent_t t1) {
  const ScanGeom g = scan_geom(batch * p->L, p->V, p->M);
  HeadArgs a;
  a.ckeys = hw.scan.chunk_keys;
  a.ctail = hw.scan.chunk_tail;
  a.cflag = hw.scan.chunk_flag;
  a.nchunks = g.nchunks;
  a.P_all = p->P_all;
  a.whh = p->whh_rm;
  a.b_hh = p->b_hh;
  a.w1 = hd.w1;
  a.w2 = hd.w2;
  a.a = hw.a;
  a.h0 = h0;
  a.states = hw.states;
  a.ghs = hw.ghs;
  a.L = p->L;
  a.M = p->M;
  a.B = p->B;
  a.k = p->k;
  a.dh = p->d_h;
  a.d_H = hd.d_H;
  a.rank = hd.rank;
  a.norm_mode = p->norm_mode;
  a.pos_offset = p->pos_offset;
  a.cost = p->cost;
  a.inv_tau = inv_tau;
  a.c2 = 1.4426950408889634f * inv_tau;
  a.out = *out;
  const size_t lds = head_lds_bytes(p->L, p->B, p->d_h, hd.rank);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&head_tree_kernel<T>),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  if (t0)
    hipExtLaunchKernelGGL(head_tree_kernel<T>, dim3(batch), dim3(kHT), lds, s, t0, t1, 0, a);
  else
    hipLaunchKernelGGL(head_tree_kernel<T>, dim3(batch), dim3(kHT), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_head(const dt_plan *p, int batch, const void *H, const dt_domino_head &hd,
                       const float *h0, float inv_tau, const HeadWorkspace &hw, dt_tree *out,
                       hipStream_t s, hipEvent_t t0, hipEvent_t t1) {
  return p->wdt == DT_BF16 ? launch_head_t<uint16_t>(p, batch, H, hd, h0, inv_tau, hw, out, s, t0, t1)
                           : launch_head_t<float>(p, batch, H, hd, h0, inv_tau, hw, out, s, t0, t1);
}

}  // namespace dt
