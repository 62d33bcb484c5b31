// Plan-time work: the vocabulary fold and weight packing.
//
// Candidate restriction (section 3.2) gathers, once per depth, the rows of the
// correction that the top-M candidates need.  Here the rows are model-only
// quantities, so they are computed once per plan for the whole vocabulary and
// every call just gathers them:
//   P[v] = W_ih E[v] + b_ih (+ b_hh on the r and z gates, which only ever
//          appear summed with it; GRU input projection of token v, 3*d_h)
//   U[v] = W_c^T E[v]         (so delta(v) = U[v] . S + c[v] = E[v] . (W_c S + b_c))
//   c[v] = E[v] . b_c
// This is one GEMM of the embedding table against the packed matrix
// [W_ih ; W_c^T] ([4 d_h, d_e], K = d_e contiguous).  bf16 weights run on the
// gfx950 bf16 MFMA (exact products, fp32 accumulation); fp32 weights use a plain
// FMA kernel.
#include "dt_internal.h"

namespace dt {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kFoldThreads = 256;
constexpr int kLdsPad = 8;  // bf16 elements of padding per LDS row

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM: block tile (WR*TI*32) x (WC*TJ*32), 4 waves as WR x WC.
// ---------------------------------------------------------------------------
template <int WR, int WC, int TI, int TJ>
__global__ __launch_bounds__(kFoldThreads) void fold_mfma_kernel(
    const uint16_t *__restrict__ emb, const int32_t *__restrict__ cand, int rows_total, int d_e,
    const uint16_t *__restrict__ wfold, int nf, int d_h, const float *__restrict__ b_ih,
    const float *__restrict__ b_c, float *__restrict__ P, float *__restrict__ U,
    float *__restrict__ cvec) {
  static_assert(WR * WC == 4, "4 waves");
  constexpr int BM = WR * TI * 32, BN = WC * TJ * 32, BK = kFoldBK;
  constexpr int LDW = BK + kLdsPad;
  __shared__ __attribute__((aligned(16))) uint16_t As[BM * LDW];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[BN * LDW];
  __shared__ float bcs[BK];
  __shared__ int32_t rowtok[BM];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave / WC, wc = wave % WC;
  const int n0 = blockIdx.x * BN, r0 = blockIdx.y * BM;
  const bool do_c = blockIdx.x == 0;  // the first column tile also computes c = E_c b_c

  for (int i = tid; i < BM; i += kFoldThreads) {
    const int r = r0 + i;
    rowtok[i] = (r < rows_total) ? (cand ? cand[r] : r) : -1;
  }
  __syncthreads();

  f32x16 acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.0f;
  float cacc = 0.0f;  // c[r] partial for rows handled by this thread (do_c only)

  constexpr int SEGS = BK / 8;  // 16-byte segments per tile row
  for (int k0 = 0; k0 < d_e; k0 += BK) {
    // global -> LDS (gathered A rows, packed B rows)
    for (int s = tid; s < BM * SEGS; s += kFoldThreads) {
      const int row = s / SEGS, seg = s % SEGS, k = k0 + seg * 8;
      uint4 v = make_uint4(0, 0, 0, 0);
      const int tok = rowtok[row];
      if (tok >= 0 && k + 8 <= d_e) v = *reinterpret_cast<const uint4 *>(emb + (size_t)tok * d_e + k);
      *reinterpret_cast<uint4 *>(&As[row * LDW + seg * 8]) = v;
    }
    for (int s = tid; s < BN * SEGS; s += kFoldThreads) {
      const int row = s / SEGS, seg = s % SEGS, k = k0 + seg * 8;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (n0 + row < nf && k + 8 <= d_e)
        v = *reinterpret_cast<const uint4 *>(wfold + (size_t)(n0 + row) * d_e + k);
      *reinterpret_cast<uint4 *>(&Bs[row * LDW + seg * 8]) = v;
    }
    if (do_c)
      for (int i = tid; i < BK; i += kFoldThreads) bcs[i] = (k0 + i < d_e) ? b_c[k0 + i] : 0.0f;
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 a[TI], b[TJ];
      const int kk = ks * 16 + (lane >> 5) * 8;
#pragma unroll
      for (int i = 0; i < TI; ++i) {
        const int row = (wr * TI + i) * 32 + (lane & 31);
        a[i] = *reinterpret_cast<const bf16x8 *>(&As[row * LDW + kk]);
      }
#pragma unroll
      for (int j = 0; j < TJ; ++j) {
        const int col = (wc * TJ + j) * 32 + (lane & 31);
        b[j] = *reinterpret_cast<const bf16x8 *>(&Bs[col * LDW + kk]);
      }
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (do_c) {
      // two threads per row, each over half of the K slice
      for (int i = tid; i < BM * 2; i += kFoldThreads) {
        const int row = i >> 1, half = i & 1;
        float s = 0.0f;
        for (int q = half * (BK / 2); q < (half + 1) * (BK / 2); ++q)
          s += bf16_to_f32(As[row * LDW + q]) * bcs[q];
        cacc += s;
      }
    }
    __syncthreads();
  }

  // epilogue: 32x32 MFMA output layout -- lane l, register q holds
  // row (q/4)*8 + (l/32)*4 + q%4, column l%32
#pragma unroll
  for (int i = 0; i < TI; ++i) {
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int col = n0 + (wc * TJ + j) * 32 + (lane & 31);
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int row = r0 + (wr * TI + i) * 32 + (q >> 2) * 8 + (lane >> 5) * 4 + (q & 3);
        if (row >= rows_total || col >= nf) continue;
        const float v = acc[i][j][q];
        if (col < 3 * d_h)
          P[(size_t)row * (3 * d_h) + col] = v + b_ih[col];
        else
          U[(size_t)row * d_h + (col - 3 * d_h)] = v;
      }
    }
  }
  static_assert(BM * 2 <= kFoldThreads, "one (row, half) pair per thread");
  if (do_c) {
    // thread tid accumulated the half-row pair i = tid; combine the two halves
    __shared__ float cpart[BM * 2];
    if (tid < BM * 2) cpart[tid] = cacc;
    __syncthreads();
    for (int row = tid; row < BM; row += kFoldThreads) {
      const int r = r0 + row;
      if (r < rows_total) cvec[r] = cpart[2 * row] + cpart[2 * row + 1];
    }
  }
}

// ---------------------------------------------------------------------------
// generic FMA path (fp32 weights, or widths the MFMA path does not take)
// ---------------------------------------------------------------------------
template <typename TW>
__device__ inline float wval(const TW *p, size_t i);
template <>
__device__ inline float wval<uint16_t>(const uint16_t *p, size_t i) {
  return bf16_to_f32(p[i]);
}
template <>
__device__ inline float wval<float>(const float *p, size_t i) {
  return p[i];
}

template <typename TW>
__global__ __launch_bounds__(256) void fold_simple_kernel(
    const TW *__restrict__ emb, const int32_t *__restrict__ cand, int rows_total, int d_e,
    const TW *__restrict__ wfold, int nf, int d_h, const float *__restrict__ b_ih,
    const float *__restrict__ b_c, float *__restrict__ P, float *__restrict__ U,
    float *__restrict__ cvec) {
  // one block per candidate row; threads over the nf+1 outputs
  const int r = blockIdx.x;
  if (r >= rows_total) return;
  const int tok = cand ? cand[r] : r;
  for (int n = threadIdx.x; n <= nf; n += blockDim.x) {
    float s = 0.0f;
    if (tok >= 0) {
      if (n < nf) {
        for (int k = 0; k < d_e; ++k)
          s += wval<TW>(emb, (size_t)tok * d_e + k) * wval<TW>(wfold, (size_t)n * d_e + k);
      } else if (b_c != nullptr) {
        for (int k = 0; k < d_e; ++k) s += wval<TW>(emb, (size_t)tok * d_e + k) * b_c[k];
      }
    }
    if (n < 3 * d_h)
      P[(size_t)r * (3 * d_h) + n] = s + b_ih[n];
    else if (n < nf)
      U[(size_t)r * d_h + (n - 3 * d_h)] = s;
    else
      cvec[r] = s;
  }
}

// ---------------------------------------------------------------------------
// plan-time packing
// ---------------------------------------------------------------------------
template <typename TW>
__global__ void pack_wfold_kernel(const TW *__restrict__ w_ih, const TW *__restrict__ w_c, int d_e,
                                  int d_h, int nf_pad, TW *__restrict__ out) {
  const size_t total = (size_t)nf_pad * d_e;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    const int n = (int)(i / d_e), k = (int)(i % d_e);
    TW v = TW(0);
    if (n < 3 * d_h)
      v = w_ih[(size_t)n * d_e + k];
    else if (n < 4 * d_h)
      v = w_c[(size_t)k * d_h + (n - 3 * d_h)];
    out[i] = v;
  }
}

template <typename TW>
__global__ void widen_kernel(const TW *__restrict__ in, int n, float *__restrict__ out) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    out[i] = in ? wval<TW>(in, i) : 0.0f;
}

// dst[i] += src[i]: folds b_hh's r and z parts into the input-side bias
__global__ void add_kernel(float *__restrict__ dst, const float *__restrict__ src, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    dst[i] += src[i];
}

// W_hh packed in MFMA A-fragment order for the expansion kernel.
// bf16 (16x16x32 MFMA): fragment (u, g, ks) is 64 lanes x 8 bf16; lane l holds
//   W_hh[g*d_h + 16u + l%16][ks*32 + (l/16)*8 + e], e = 0..7.
// fp32 (16x16x4 MFMA, four per k-group of 16): fragment (u, g, q) is 64 lanes x 4
//   floats; lane l holds W_hh[g*d_h + 16u + l%16][16q + (l/16)*4 + e], e = 0..3.
__global__ void pack_whh_bf16_kernel(const uint16_t *__restrict__ w_hh, int d_h,
                                     uint16_t *__restrict__ out) {
  const int nks = d_h / 32;
  const size_t total = (size_t)3 * d_h * d_h;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    const int e = (int)(i % 8);
    const int lane = (int)((i / 8) % 64);
    const size_t frag = i / 512;
    const int ks = (int)(frag % nks);
    const int g = (int)((frag / nks) % 3);
    const int u = (int)(frag / nks / 3);
    const int row = g * d_h + 16 * u + (lane & 15);
    const int k = ks * 32 + (lane >> 4) * 8 + e;
    out[i] = w_hh[(size_t)row * d_h + k];
  }
}

__global__ void pack_whh_f32_kernel(const float *__restrict__ w_hh, int d_h, float *__restrict__ out) {
  const int nq = d_h / 16;
  const size_t total = (size_t)3 * d_h * d_h;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    const int e = (int)(i % 4);
    const int lane = (int)((i / 4) % 64);
    const size_t frag = i / 256;
    const int q = (int)(frag % nq);
    const int g = (int)((frag / nq) % 3);
    const int u = (int)(frag / nq / 3);
    const int row = g * d_h + 16 * u + (lane & 15);
    const int k = 16 * q + (lane >> 4) * 4 + e;
    out[i] = w_hh[(size_t)row * d_h + k];
  }
}

inline int grid_for(size_t n) {
  size_t b = (n + 255) / 256;
  return (int)(b > 65535 ? 65535 : (b < 1 ? 1 : b));
}

}  // namespace

hipError_t pack_weights(dt_model *p, const dt_gru *gru, const dt_head *head, hipStream_t s) {
  const int d_e = p->d_e, d_h = p->d_h;
  const size_t wfold_n = (size_t)p->nf_pad * d_e;
  if (p->wdt == DT_BF16) {
    hipLaunchKernelGGL(pack_wfold_kernel<uint16_t>, dim3(grid_for(wfold_n)), dim3(256), 0, s,
                       (const uint16_t *)gru->w_ih, (const uint16_t *)head->w, d_e, d_h, p->nf_pad,
                       (uint16_t *)p->wfold);
    hipLaunchKernelGGL(widen_kernel<uint16_t>, dim3(grid_for(3 * d_h)), dim3(256), 0, s,
                       (const uint16_t *)gru->b_ih, 3 * d_h, p->b_ih);
    hipLaunchKernelGGL(widen_kernel<uint16_t>, dim3(grid_for(3 * d_h)), dim3(256), 0, s,
                       (const uint16_t *)gru->b_hh, 3 * d_h, p->b_hh);
    hipLaunchKernelGGL(widen_kernel<uint16_t>, dim3(grid_for(d_e)), dim3(256), 0, s,
                       (const uint16_t *)head->b, d_e, p->b_c);
    hipLaunchKernelGGL(pack_whh_bf16_kernel, dim3(grid_for((size_t)3 * d_h * d_h)), dim3(256), 0,
                       s, (const uint16_t *)gru->w_hh, d_h, (uint16_t *)p->whh_t);
  } else {
    hipLaunchKernelGGL(pack_wfold_kernel<float>, dim3(grid_for(wfold_n)), dim3(256), 0, s,
                       (const float *)gru->w_ih, (const float *)head->w, d_e, d_h, p->nf_pad,
                       (float *)p->wfold);
    hipLaunchKernelGGL(widen_kernel<float>, dim3(grid_for(3 * d_h)), dim3(256), 0, s,
                       (const float *)gru->b_ih, 3 * d_h, p->b_ih);
    hipLaunchKernelGGL(widen_kernel<float>, dim3(grid_for(3 * d_h)), dim3(256), 0, s,
                       (const float *)gru->b_hh, 3 * d_h, p->b_hh);
    hipLaunchKernelGGL(widen_kernel<float>, dim3(grid_for(d_e)), dim3(256), 0, s,
                       (const float *)head->b, d_e, p->b_c);
    hipLaunchKernelGGL(pack_whh_f32_kernel, dim3(grid_for((size_t)3 * d_h * d_h)), dim3(256), 0, s,
                       (const float *)gru->w_hh, d_h, (float *)p->whh_t);
  }
  hipLaunchKernelGGL(add_kernel, dim3(grid_for(2 * d_h)), dim3(256), 0, s, p->b_ih, p->b_hh, 2 * d_h);
  return hipGetLastError();
}

hipError_t fold_vocab(const dt_model *p, hipStream_t s) {
  const int rows_total = p->V;
  const float *bc = p->b_c;  // zeros when the head has no bias
  if (p->wdt == DT_BF16 && p->d_e % 8 == 0) {
    const int ntile_n = (p->nf + 127) / 128;
    dim3 grid(ntile_n, (rows_total + 127) / 128);
    hipLaunchKernelGGL((fold_mfma_kernel<2, 2, 2, 2>), grid, dim3(kFoldThreads), 0, s,
                       (const uint16_t *)p->emb, nullptr, rows_total, p->d_e,
                       (const uint16_t *)p->wfold, p->nf, p->d_h, p->b_ih, bc, p->P_all, p->U_all,
                       p->c_all);
  } else if (p->wdt == DT_BF16) {
    hipLaunchKernelGGL(fold_simple_kernel<uint16_t>, dim3(rows_total), dim3(256), 0, s,
                       (const uint16_t *)p->emb, nullptr, rows_total, p->d_e,
                       (const uint16_t *)p->wfold, p->nf, p->d_h, p->b_ih, bc, p->P_all, p->U_all,
                       p->c_all);
  } else {
    hipLaunchKernelGGL(fold_simple_kernel<float>, dim3(rows_total), dim3(256), 0, s,
                       (const float *)p->emb, nullptr, rows_total, p->d_e, (const float *)p->wfold,
                       p->nf, p->d_h, p->b_ih, bc, p->P_all, p->U_all, p->c_all);
  }
  return hipGetLastError();
}

}  // namespace dt
