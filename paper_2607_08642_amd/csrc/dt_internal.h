// Internal definitions shared by the HIP sources of libdominotree (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <atomic>

#include "dominotree.h"

namespace dt {

// ---------------------------------------------------------------------------
// limits (the public envelope is documented in dominotree.h)
// ---------------------------------------------------------------------------
constexpr int kMaxM = 256;
constexpr int kMaxB = 256;
constexpr int kMaxL = 64;
constexpr int kMaxDh = 1024;
constexpr int kMaxDe = 8192;

// scan: one workgroup of 256 threads per (row, chunk of kScanChunk elements)
constexpr int kScanThreads = 256;
constexpr int kScanPerThread = 40;                         // elements held per thread
constexpr int kScanChunk = kScanThreads * kScanPerThread;  // 10240
constexpr int kScanSortCap = 4096;   // bitonic sort buffer (keys) per workgroup
constexpr int kScanSlots = 1024;    // scan workgroups resident at once (4 per CU of 256)
constexpr int kScanFlushAt = 256;    // fallback: flush the candidate buffer beyond this
constexpr int kMergeLdsMax = 96 * 1024;  // row merge buffer (sel::merge_buf_bytes) at most

// fold GEMM tile (bf16 MFMA path)
constexpr int kFoldBM = 128;
constexpr int kFoldBN = 128;
constexpr int kFoldBK = 64;

// expansion kernel
constexpr int kExpThreads = 512;
constexpr int kNodeCap = 1536;       // live nodes per tree kept in LDS
constexpr int kChunkNodes = 16;      // nodes expanded together (shared weight pass)
constexpr int kBarStride = 64;       // ints per tree of barrier counters (own cache lines)
constexpr int kMaxXcd = 8;           // XCDs with a member-slot counter each
constexpr int kSlotStride = 32;      // ints per XCD's slot counter (its own 128-byte line)
constexpr int kSlotRows = kMaxXcd * kSlotStride / kBarStride;  // kBarStride rows of slot counters
constexpr int kProfSlots = 1024;     // profiled calls kept for stage averages

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ---------------------------------------------------------------------------
// order-preserving 64-bit keys: (value desc, index asc) <=> key desc.
// high word: IEEE bits mapped to an unsigned order (-0 folded onto +0);
// low word: bitwise NOT of the index.  Key 0 is never produced (sentinel).
// ---------------------------------------------------------------------------
__host__ __device__ inline uint32_t ordered_bits(float v) {
  uint32_t u;
  if (v == 0.0f) v = 0.0f;
  __builtin_memcpy(&u, &v, 4);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__host__ __device__ inline float ordered_to_float(uint32_t o) {
  uint32_t u = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
  float v;
  __builtin_memcpy(&v, &u, 4);
  return v;
}
__host__ __device__ inline uint64_t make_key(float v, uint32_t idx) {
  return ((uint64_t)ordered_bits(v) << 32) | (uint32_t)(~idx);
}
__host__ __device__ inline float key_value(uint64_t k) { return ordered_to_float((uint32_t)(k >> 32)); }
__host__ __device__ inline uint32_t key_index(uint64_t k) { return ~(uint32_t)k; }

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// ---------------------------------------------------------------------------
// plan
// ---------------------------------------------------------------------------
struct ScanGeom {
  int rows, V, M;
  int chunk;    // elements per segment (a multiple of kScanChunk)
  int nchunks;  // segments (= sorted lists) per row
};

}  // namespace dt

// The model-level tables: the vocabulary folded through the GRU input
// projection and the correction head, and the repacked weights.  Shared by
// every plan created from the model; freed with the last reference.
struct dt_model {
  int V, d_e, d_h, wdt;
  const void *emb;
  void *wfold;      // [nf_pad, d_e] (weights dtype): rows [0,3dh) = W_ih, [3dh,4dh) = W_c^T;
                    // only alive while the model is created
  float *P_all;     // [V][3dh]  W_ih E[v] + b_ih + (b_hh on gates r, z)
  float *U_all;     // [V][dh]   W_c^T E[v]
  float *c_all;     // [V]       E[v] . b_c
  int nf, nf_pad;   // nf = 4*d_h
  float *b_ih;      // [3dh] fp32 b_ih + (b_hh on gates r, z); zeros when absent
  float *b_hh;      // [3dh] fp32
  float *b_c;       // [d_e] fp32 (zeros when absent)
  int has_bc;
  void *whh_t;      // W_hh in MFMA A-fragment order (see pack_whh_*_kernel)
  void *whh_rm;     // [3dh][dh] W_hh as given (weights dtype), for the Domino-head path
  int device;       // the device its memory lives on
  std::atomic<int> refs;  // the creator's reference plus one per plan
};

struct dt_plan {
  int V, d_e, d_h, L, M, B, k, norm_mode, pos_offset, scorer;
  int wdt, ldt, max_batch;
  dt_model *model;  // the tables below are the model's (one reference held)
  const float *P_all, *U_all, *c_all, *b_ih, *b_hh;
  const void *whh_t, *whh_rm;
  int num_cus;
  int num_xcd;              // XCDs of the device (workgroups are dealt to them round-robin)
  size_t max_lds;           // LDS bytes a workgroup may allocate on the device
  int frontier_w;           // dt_options.frontier_width (0: the heap builder)
  int spin_limit;           // dt_options.debug_spin_limit (0: the default)
  int device;               // the device the plan was created on (its memory lives there)
  int profiling;            // > 0: record stage events on every profiling-th dt_build_tree call
  int calls_since;          // dt_build_tree calls since profiling was enabled
  int profiled_calls;       // calls recorded since profiling was enabled
  hipEvent_t *ev;           // [kProfSlots][4] start and end of both kernels, one slot per call (ring)
  float *cost;              // adaptive budget (dt_plan_set_adaptive_budget): [B + 2] device
                            // floats C_d, C_v(0..B); null = fixed budget
  float *cost_buf;          // its buffer (allocated on first use, freed with the plan)
  int32_t *stats;           // [max_batch][2] expansion steps and expanded nodes of the last
                            // profiled call (device; allocated when profiling is enabled)
  int stats_batch;          // trees of the last profiled call
};

namespace dt {

struct Workspace {
  // scan
  uint64_t *chunk_keys;   // [rows][nchunks][M]
  float2 *chunk_tail;     // [rows][nchunks] (max, sum of exp((x-max)/tau))
  int32_t *chunk_flag;    // [rows][nchunks]
  int32_t *cand;          // [rows][M]
  float *candv;           // [rows][M]
  float *tail;            // [rows]
  int32_t *row_flag;      // [rows]
  // expansion
  float *states;          // [batch][ecap][dh]
  float *part;            // [batch][2][G][16][MP] partial corrections
  int32_t *bar;           // [2][batch + kSlotRows][kBarStride] barrier and slot counters (one set
                          // per expansion launch of a call)
  float *menus;           // [batch][L][MP] corrected menus of the greedy chain (scorer
                          // DT_SCORER_STATIC)
  int ecap;
  size_t bytes;
};

ScanGeom scan_geom(int rows, int V, int M);
size_t merge_lds_bytes(const ScanGeom &g);  // LDS of the per-row merge (<= kMergeLdsMax)
size_t scan_bytes(const ScanGeom &g);
// carve the scan part of a workspace; returns bytes used
size_t carve_scan(char *base, const ScanGeom &g, Workspace *ws);
Workspace carve(const dt_plan *p, int batch, char *base);

// kernel launchers (return hipError_t of the launch)
// Domino's head: a[row][r] = W_1^H H_row over the launch's rows, computed by
// `extra` more workgroups per row of the scan launch
struct HeadProj {
  const void *w1, *H;  // [rank][ld1], [rows][d_H] (weights dtype wdt)
  float *a;            // [rows][rank]
  int d_H, ld1, rank, wdt, extra;
};
HeadProj head_proj_args(const dt_plan *p, int rows, const void *H, const dt_domino_head &hd, float *a_out);
// kernel launchers; with t0/t1 the launch records HIP events at the kernel's
// start and end (hipExtLaunchKernel), used for stage timing
hipError_t launch_scan_chunks(const void *logits, int ldt, const ScanGeom &g, float inv_tau,
                              const Workspace &ws, int32_t *zero_ptr, int zero_n, hipStream_t s,
                              hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr,
                              const HeadProj *hp = nullptr);
hipError_t launch_scan_merge(const ScanGeom &g, float inv_tau, const Workspace &ws, hipStream_t s);
hipError_t fold_vocab(const dt_model *m, hipStream_t s);
// Domino-head path (dt_build_tree_head): heap entries per tree, workspace, launch
constexpr int kHeadCap = 4096;
struct HeadWorkspace {
  Workspace scan;  // scan segment lists (chunk_keys, chunk_tail, chunk_flag) and row arrays
  float *a;        // [batch * L][rank] W_1^H H
  float *states;   // [batch][B + 1][dh]
  float *ghs;      // [batch][B + 1][3dh]
  size_t bytes;
};
HeadWorkspace carve_head(const dt_plan *p, int batch, int rank, char *base);
size_t head_lds_bytes(int L, int B, int dh, int rank);
// (with t0/t1: events at the start and end of the tree kernel)
hipError_t launch_head(const dt_plan *p, int batch, const void *H, const dt_domino_head &hd,
                       const float *h0, float inv_tau, const HeadWorkspace &hw, dt_tree *out,
                       hipStream_t s, hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr);
// Domino's own head on the expansion kernel: its tensors for one launch
struct HeadIn {
  const void *w1, *w2;  // [rank][d_H + d_h], [V][rank] (weights dtype)
  const float *a;       // [batch * L][rank] a_d = W_1^H H_d
  float *hpart;         // [batch][2][G][16][rank] workspace
  int rank, d_H;
};
// One expansion launch: DominoTree (the default), or, for the ablation arms,
// without the correction (nocorr: the marginals, or menu_in's per-depth menus)
// and/or writing every expanded depth's menu (menu_out; the greedy chain), or
// with Domino's own head in place of the linear one (head).
struct ExpMode {
  int nocorr = 0;                 // no GRU, no correction, no exchange
  const float *menu_in = nullptr;  // [batch][L][MP] normalised log-probs of each depth's slots
  float *menu_out = nullptr;       // written from every expanded node (a chain: one per depth)
  int emit = 1;                   // 0: no replay or emission (outputs untouched)
  int skip_merge = 0;             // the rows were merged by an earlier launch of the call
  int k = 0, B = 0;               // 0: the plan's
  int32_t *bar = nullptr;         // this launch's counters (zeroed), nullptr: ws.bar
  int32_t *stats = nullptr;       // [batch][2] steps and expanded nodes per tree (profiling)
  const HeadIn *head = nullptr;   // Domino's own head in place of the linear one
};
hipError_t launch_expand(const dt_plan *p, int batch, const float *h0, float inv_tau,
                         const Workspace &ws, const dt_tree *out, hipStream_t s,
                         hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr,
                         const ExpMode &mode = ExpMode());
// members per tree: the largest power of two (<= 16) that leaves each member a
// multiple of 16 and at least 32 hidden units, fits the grid (every XCD holding
// the same number of tree slots) one workgroup per CU, and whose LDS layout fits
// max_lds
int expand_group_size(int d_h, int num_cus, int num_xcd, int batch, int M, int L, int nchunks,
                      size_t max_lds);
int expand_group_size(const dt_plan *p, int batch);
size_t expand_lds_bytes(int dh, int G, int M, int nchunks, int L, int rj = 0, int wbytes = 0);
size_t expand_part_bytes(const dt_plan *p, int batch);
hipError_t pack_weights(dt_model *m, const dt_gru *gru, const dt_head *head, hipStream_t s);

}  // namespace dt
