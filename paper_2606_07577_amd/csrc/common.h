// Internal declarations shared by the library's HIP translation units.
// Target: gfx950 (CDNA4) only: 64-lane wavefronts, MFMA 32x32 tiles.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

namespace omnimem {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Device copy of one layer's working-set descriptor.  Strides in elements.
struct LayerDesc {
  const void* q;
  const void* k;
  const void* v;
  const uint8_t* mod;
  const float* lse_in;   // caller-supplied log-sum-exp [H_q][n_chunk] or null
  void* k_out;
  void* v_out;
  int64_t q_hs, q_rs;
  int64_t kv_hs, kv_rs;
  int64_t out_hs, out_rs;
  int32_t n_cache, n_chunk, n;
  float scale_log2;      // softmax scale times log2(e)
  // Work layout of the two score passes (see PassPlan): the layer's first
  // tile in each pass's global tile sequence and its tiles per query head.
  int64_t lse_base, cs_base;
  int32_t lse_th, cs_th;
  int64_t lse_rbase, cs_rbase;  // the layer's first row in each pass
  const void* hidden;           // [N][dh] hidden states (redundancy source 2)
  void* hidden_out;             // kept rows' hidden states, or null
  int64_t hidden_rs, hidden_out_rs;
  uint8_t* mod_out;             // modality of the kept rows, or null
  int32_t out_cap;              // rows per head of k_out / v_out
  int32_t inplace;              // 1: k_out, v_out are k, v (compaction in place)
  // omnimem_append only: the layer's new chunk rows.
  const void* ck;
  const void* cv;
  const uint8_t* cmod;
  int64_t c_hs, c_rs;
};

// Sizes fixed for a context.
struct Dims {
  int L, Hq, Hkv, G, d;
  int64_t max_tokens, max_chunk;
  int causal;
  int qb;       // 256-query blocks covering max_chunk
  int kb;       // 256-key blocks covering max_tokens
  int dh;       // hidden-state width (0: none)
};

// Score-pass work decomposition.  A "row" is one 256-row block that a
// workgroup keeps in registers (LSE pass: queries of one head; column-sum
// pass: keys of one query head); its "tiles" are the 64-row tiles it streams
// past them (LSE: visible key tiles; column sums: query tiles that see a
// key of the block).  Rows are numbered layer-major, then head, then block,
// and their tiles form one global sequence of W tiles, cut into chunks of c
// tiles.  Workgroup i of P takes chunks i, i + P, i + 2P, ...: at any time
// the P workgroups work on one stretch of the sequence (so the streamed
// operands of the few heads in it stay in L2), and the work per workgroup
// differs by at most one chunk.  A chunk may hold parts of several rows;
// each part writes a partial result for (row, segment), the segment being
// the chunk's index minus that of the row's first tile.  c is at least
// (longest row) / (kMaxSeg - 1), so no row has more than kMaxSeg segments.
// With many more rows than workgroup slots a plan has c = 0 ("row mode"):
// one workgroup per row, W = the number of rows, and a single segment.
constexpr int kScoreBlock = 256;  // rows a workgroup keeps in registers
constexpr int kScoreTile = 64;    // rows per streamed tile
constexpr int kMaxSeg = 4;
constexpr int kGatherRows = 64;   // slots per tile (and workgroup) of the in-place gather and its staging
struct PassPlan {
  int64_t W;  // tiles
  int P;      // workgroups
  int c;      // tiles per chunk
};
// Segment of the row starting at tile `start` that holds tile g.
__host__ __device__ inline int plan_seg(const PassPlan& p, int64_t start, int64_t g) {
  return p.c == 0 ? 0 : (int)(g / p.c - start / p.c);
}
// LSE pass: key tiles seen by the queries [256 b, 256 b + 256).
__host__ __device__ inline int lse_row_tiles(int N, int nc, int C, int b, int causal) {
  const int q0 = b * kScoreBlock;
  if (q0 >= C) return 0;
  const int kend = causal ? std::min(N, nc + std::min(q0 + kScoreBlock, C)) : N;
  return (kend + kScoreTile - 1) / kScoreTile;
}
// Column-sum pass: first query tile that sees a key of [256 b, 256 b + 256)
// and the number of query tiles from there.
__host__ __device__ inline int cs_first_tile(int nc, int b, int causal) {
  return causal ? std::max(0, b * kScoreBlock - nc) / kScoreTile : 0;
}
__host__ __device__ inline int cs_row_tiles(int N, int nc, int C, int b, int causal) {
  if (b * kScoreBlock >= N) return 0;
  return std::max(0, (C + kScoreTile - 1) / kScoreTile - cs_first_tile(nc, b, causal));
}

// Loads through the global address space.  Pointers read from a
// descriptor are generic; a generic (flat) load also counts against the LDS
// wait counter, which would make every LDS wait wait for HBM as well.
template <typename T>
__device__ inline T gload(const void* p) {
  typedef const __attribute__((address_space(1))) T global_t;
  return *(global_t*)(p);
}
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ inline uint4 gload16(const void* p) {
  const u32x4 v = gload<u32x4>(p);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// Index of the calling wavefront in its workgroup, as a scalar.
__device__ inline int wave_id() { return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)); }
// A value that is the same in every lane (read from LDS, say), kept in a
// scalar register.
__device__ inline int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// ---------------------------------------------------------------------------
// MFMA operand traits.  A 32x32 output tile D[M][N] += A[M][k] B[k][N] is
// computed in k-steps; lane l supplies row (l & 31) of A (and column (l & 31)
// of B), holding PER_LANE consecutive k-elements starting at
// ks*KSTEP + (l >> 5)*PER_LANE.  The output element held in accumulator
// register r of lane l is D[(r >> 2)*8 + (l >> 5)*4 + (r & 3)][l & 31].
// ---------------------------------------------------------------------------
template <typename T> struct Mfma;

template <> struct Mfma<uint16_t> {  // bf16 storage, v_mfma_f32_32x32x16_bf16
  static constexpr int KSTEP = 16;
  static constexpr int PER_LANE = 8;
  using frag = bf16x8;
  __device__ static inline floatx16 mma(frag a, frag b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static inline frag load(const uint16_t* p) {
    return *reinterpret_cast<const frag*>(p);
  }
  __device__ static inline frag gload(const uint16_t* p) { return omnimem::gload<frag>(p); }
  __device__ static inline frag zero() { return frag{}; }
};

template <> struct Mfma<float> {  // fp32, v_mfma_f32_32x32x2_f32
  static constexpr int KSTEP = 2;
  static constexpr int PER_LANE = 1;
  using frag = float;
  __device__ static inline floatx16 mma(frag a, frag b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  __device__ static inline frag load(const float* p) { return *p; }
  __device__ static inline frag gload(const float* p) { return omnimem::gload<float>(p); }
  __device__ static inline frag zero() { return 0.0f; }
};

// Workgroups are dispatched to the 8 XCDs round robin (block b on XCD
// b % 8).  With the grid padded to a multiple of 8, this bijection maps
// consecutive logical ids onto the same XCD, so workgroups that share data
// share one L2.
constexpr int kXcds = 8;
__host__ __device__ inline unsigned xcd_grid(int64_t logical_blocks) {
  return (unsigned)((logical_blocks + kXcds - 1) / kXcds * kXcds);
}
__device__ inline int xcd_swizzle(unsigned b, unsigned grid) {
  return (int)((b % kXcds) * (grid / kXcds) + b / kXcds);
}

// Row of the 32x32 output tile held by accumulator register r of lane l.
__device__ inline int acc_row(int r, int lane) { return (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3); }

// LDS row padding: 16 bytes keeps ds_read_b128 of consecutive rows on
// different banks.
template <typename T> constexpr int lds_pad() { return 16 / (int)sizeof(T); }

// Copy `rows` rows of D elements from global (row r at src + r*row_stride)
// into an LDS tile with row stride D + pad; rows at or past `valid` are
// zero-filled.  Every thread of the block takes part.
template <typename T, int D>
__device__ inline void stage_rows(T* lds, const T* src, int64_t row_stride, int rows, int valid) {
  constexpr int CPR = D * (int)sizeof(T) / 16;  // 16-byte chunks per row
  constexpr int LD = D + lds_pad<T>();
  for (int c = threadIdx.x; c < rows * CPR; c += blockDim.x) {
    const int r = c / CPR, x = c % CPR;
    uint4 val = make_uint4(0, 0, 0, 0);
    if (r < valid) val = gload16(src + (int64_t)r * row_stride + x * (16 / sizeof(T)));
    *reinterpret_cast<uint4*>(lds + r * LD + x * (16 / sizeof(T))) = val;
  }
}

// Same, with an explicit row list (gathered rows).
template <typename T, int D>
__device__ inline void stage_rows_gather(T* lds, const T* base, int64_t row_stride, const int* rows_idx,
                                         int rows, int valid) {
  constexpr int CPR = D * (int)sizeof(T) / 16;
  constexpr int LD = D + lds_pad<T>();
  for (int c = threadIdx.x; c < rows * CPR; c += blockDim.x) {
    const int r = c / CPR, x = c % CPR;
    uint4 val = make_uint4(0, 0, 0, 0);
    if (r < valid) val = gload16(base + (int64_t)rows_idx[r] * row_stride + x * (16 / sizeof(T)));
    *reinterpret_cast<uint4*>(lds + r * LD + x * (16 / sizeof(T))) = val;
  }
}

// Order-preserving map float -> int32 (signed compare), an involution.
__device__ inline int ord_f32(float f) {
  int i = __float_as_int(f);
  return i ^ ((i >> 31) & 0x7fffffff);
}
__device__ inline float unord_f32(int i) { return __int_as_float(i ^ ((i >> 31) & 0x7fffffff)); }

constexpr int kNoPartner = (int)0x80000000;  // below ord_f32 of every float

// The modality row lists hold max_tokens entries plus kListPad more after
// each list's end, set to the list's last row: a 64-row tile or a 256-row
// register block that runs past a segment's end reads valid rows.
constexpr int kListPad = 256;
__host__ __device__ inline int64_t list_stride(int64_t max_tokens) { return max_tokens + kListPad; }

// Top-k split over several workgroups per (layer, KV head): rows are taken
// in slices of kTopkSlice; the keys and candidate arrays of a (layer, KV
// head) are max_tokens rounded up to whole slices; at most kTopkMaxSlices
// slices per working set (larger contexts use the one-workgroup top-k).
constexpr int kTopkSlice = 2048;
constexpr int kTopkMaxSlices = 256;
constexpr int kTopkBins = 4096;   // bins of the first two radix digits
__host__ __device__ inline int64_t topk_stride(int64_t max_tokens) {
  return (max_tokens + kTopkSlice - 1) / kTopkSlice * kTopkSlice;
}

// ---------------------------------------------------------------------------
// Optional launch timing (see omnimem_profile).
// ---------------------------------------------------------------------------
enum KernelId {
  K_LSE, K_LSE_MERGE, K_COLSUM, K_HEADSUM, K_LISTS, K_NORMS, K_GRAM, K_GRAM_FINISH, K_ADJ,
  K_AVBA_PART, K_AVBA_ALLOC, K_TOPK, K_GATHER, K_GATHER_H, K_ADJ_H, K_NORMS_H, K_GRAM_H, K_FINISH_H, K_LAYER_IN,
  K_STAGE, K_GATHER_IP, K_APPEND, K_GRAM_SYM, K_TOPK_HIST, K_TOPK_BIN, K_TOPK_EMIT, K_TOPK_REG, K_COUNT
};
struct Profiler;
void prof_mark(Profiler* p, int kernel, hipStream_t st, bool begin);

// Launch `stmt` bracketed by profiler events when profiling is on.
#define OMNIMEM_LAUNCH(ws, kid, st, ...)                 \
  do {                                                   \
    if ((ws).prof) prof_mark((ws).prof, (kid), (st), true); \
    __VA_ARGS__;                                         \
    if ((ws).prof) prof_mark((ws).prof, (kid), (st), false); \
  } while (0)

// ---------------------------------------------------------------------------
// Workspace owned by a context (device pointers), sized at creation.
// ---------------------------------------------------------------------------
struct Workspace {
  LayerDesc* desc;        // [slots][L]
  float2* lse_part;       // [L][Hq][qb][kMaxSeg][256] partial (reference, sum) in log2 units
  float* lse2;            // [L][Hq][max_chunk] merged normaliser, log2 units
  float* part;            // [L][Hq][kb][kMaxSeg][256] partial column sums per query head
  int* pos;               // [L][2][max_tokens + kListPad] visual rows, audio rows (ascending)
  int* rank;              // [L][max_tokens]  rank of row j inside its modality
  int* counts;            // [L][2]           K_v, K_a
  float* inv_norm;        // [L][Hkv][max_tokens] inverse norms, segment order
  int* best;              // [L][Hkv][max_tokens] ord_f32 of the best cosine, segment order
  void* perm;             // fp32 only: [L][Hkv][max_tokens][d] rows in segment order (visual, then audio)
  int gram_grid;          // persistent Gram workgroups
  double* stat_part;      // [L][Hkv][chunks][2][4]
  double* calib;          // [L] sums of C^(l) over the calibration steps
  int* eff;               // [L][2] budgets as applied by select
  int* idx;               // [L][Hkv][max_tokens] fallback for the idx output
  uint32_t* keys;         // [L][Hkv][topk_stride(max_tokens)]
  // Split top-k (see topk_hist / topk_bin / topk_emit).
  int* tk_hist;           // [L][Hkv][2][kTopkBins] first-digit histograms; all zero between calls
  int* tk_seg;            // [L][Hkv][2][8] per modality: mode, bin, need, count, M, first slot, K
  int* tk_slice;          // [L][Hkv][kTopkMaxSlices][2] per slice: keys above the bin, visual and audio
  uint2* tk_cand;         // [L][Hkv][topk_stride(max_tokens)] candidates (key, row): visual from the
                          // front, audio from the back
  int* tk_ccount;         // [L][Hkv][2] candidates listed so far (cleared by each call's first kernel)
  float* layer_as;        // [2][L][max_tokens] layer-shared selection inputs (null without it)
  // In-place compaction (null / 0 unless the context reserves staging rows).
  int stage_rows;         // staging rows per (layer, KV head)
  void* stage;            // [2][L][Hkv][stage_rows][d] staged K, then V rows
  int* slot_of;           // [L][Hkv][max_tokens] slot that reads row j (-1: dropped)
  int* read_flags;        // [L][Hkv][tiles] 1 once a kGatherRows-slot tile has read its rows
  int* ctl;               // [1] this call's staging need beyond the reserve (0: none), [2] largest need
                          // and [3] wait time-outs since the last query ([0] unused)
  int* tickets;           // [L * Hkv][32] tile tickets of the in-place gather, one 128-byte line each
  Profiler* prof;         // null unless timing is on
};

// Launchers (each returns hipGetLastError() after its launches).
hipError_t launch_score(const Dims& dm, int dtype, const LayerDesc* desc, const Workspace& ws,
                        const PassPlan& lse_plan, const PassPlan& cs_plan, float* lse_out, float* a,
                        hipStream_t st);
void plan_score(const Dims& dm, LayerDesc* layers, int max_workgroups, PassPlan* lse_plan, PassPlan* cs_plan);
int allocate_part_chunks(const Dims& dm);
hipError_t launch_redundancy(const Dims& dm, int dtype, int sim, int on_keys, const LayerDesc* desc,
                             const Workspace& ws, float* s, hipStream_t st);
hipError_t launch_lists(const Dims& dm, const LayerDesc* desc, const Workspace& ws, hipStream_t st);
hipError_t launch_allocate(const Dims& dm, const LayerDesc* desc, const Workspace& ws,
                           const float* a, const float* s, int64_t total, float ratio_r,
                           float temperature, float bmin_frac, float bmax_frac, int32_t* budgets,
                           float* stats, hipStream_t st);
hipError_t launch_calibrate(const Dims& dm, const LayerDesc* desc, const Workspace& ws, const float* a,
                            const float* s, float ratio_r, bool first, float* stats, hipStream_t st);
hipError_t launch_calibration_budgets(const Dims& dm, const Workspace& ws, int64_t total, float temperature,
                                      float bmin_frac, float bmax_frac, int steps, int32_t* layer_budgets,
                                      hipStream_t st);
hipError_t launch_allocate_fixed(const Dims& dm, const LayerDesc* desc, const Workspace& ws, const float* a,
                                 const float* s, const int32_t* layer_budgets, float ratio_r, int32_t* budgets,
                                 float* stats, hipStream_t st);
hipError_t launch_select_compact(const Dims& dm, int dtype, float lambda, int shared, bool hidden, int inplace,
                                 int max_n, int topk_path, const LayerDesc* desc, const Workspace& ws,
                                 const float* a, const float* s, const int32_t* budgets, int32_t* idx,
                                 hipStream_t st);  // inplace: 0 none, 1 some, 2 all; max_n: largest N;
                                                   // topk_path: an omnimem_topk_path other than AUTO
// Rows up to which the top-k can keep every key in registers, and the
// largest working set the split top-k takes.
constexpr int kTopkRegRows = 8192;
constexpr int64_t kTopkSplitMaxRows = (int64_t)kTopkMaxSlices * kTopkSlice;
hipError_t launch_append(const Dims& dm, int dtype, const LayerDesc* desc, const Workspace& ws, int64_t max_rows,
                         hipStream_t st);

// One LDS stage of kScoreTile rows of D elements, unpadded.  The 16-byte chunk c
// of row r is stored at chunk position c ^ (r & XM): the 16 rows that a
// quarter-wave reads at the same chunk land on 16 different bank groups.
// Rows are copied by the global-to-LDS DMA path (global_load_lds_dwordx4),
// which writes 16 bytes per lane at consecutive LDS slots: no registers and
// no LDS store instructions.
template <typename T, int D>
struct SwzTile {
  static constexpr int ROWB = D * (int)sizeof(T);   // bytes per row
  static constexpr int CPR = ROWB / 16;             // chunks per row
  static constexpr int XM = (CPR < 16 ? CPR : 16) - 1;
  static constexpr int EPC = 16 / (int)sizeof(T);   // elements per chunk
  static constexpr int ELEMS = kScoreTile * D;
  static constexpr int INSTR_PER_WAVE = kScoreTile * CPR / 64 / 4;  // 1 KB copies per wave

  // Byte offset of element e of row r.
  __device__ static inline int off(int r, int e) {
    return r * ROWB + (((e / EPC) ^ (r & XM)) << 4) + (e % EPC) * (int)sizeof(T);
  }
  // Copy rows src[0 .. kScoreTile) (rows at or past `valid` >= 1 repeat row
  // valid - 1) into `lds`.  Every thread of the block takes part.
  __device__ static inline void dma(T* lds, const T* src, int64_t row_stride, int valid) {
    const int w = wave_id(), ln = threadIdx.x & 63;
#pragma unroll
    for (int j = 0; j < INSTR_PER_WAVE; ++j) {
      const int J = w * INSTR_PER_WAVE + j;
      const int slot = J * 64 + ln;
      const int row = slot / CPR, pos = slot % CPR;
      const int c = pos ^ (row & XM);
      const T* g = src + (int64_t)min(row, valid - 1) * row_stride + c * EPC;
      __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)g,
                                       (__attribute__((address_space(3))) void*)(lds + J * 64 * EPC), 16, 0, 0);
    }
  }
  // Per-lane byte offsets of the copies of a full tile, computed once: a
  // full tile's copies then cost no address arithmetic beyond a scalar base.
  struct Plan {
    uint32_t off[INSTR_PER_WAVE];
    bool ok;  // offsets fit in 31 bits
  };
  __device__ static inline Plan plan(int64_t row_stride) {
    Plan p;
    p.ok = (int64_t)kScoreTile * row_stride * (int64_t)sizeof(T) < (int64_t{1} << 31);
    const int w = wave_id(), ln = threadIdx.x & 63;
#pragma unroll
    for (int j = 0; j < INSTR_PER_WAVE; ++j) {
      const int slot = (w * INSTR_PER_WAVE + j) * 64 + ln;
      const int row = slot / CPR, c = (slot % CPR) ^ (row & XM);
      p.off[j] = (uint32_t)(((int64_t)row * row_stride + c * EPC) * (int64_t)sizeof(T));
    }
    return p;
  }
  // dma() for a tile of `valid` rows, through the plan when the tile is full.
  __device__ static inline void copy(T* lds, const T* src, int64_t row_stride, int valid, const Plan& p) {
    if (valid >= kScoreTile && p.ok) {
      const int w = wave_id();
#pragma unroll
      for (int j = 0; j < INSTR_PER_WAVE; ++j) {
        const int J = w * INSTR_PER_WAVE + j;
        const char* g = reinterpret_cast<const char*>(src) + p.off[j];
        __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)g,
                                         (__attribute__((address_space(3))) void*)(lds + J * 64 * EPC), 16, 0, 0);
      }
    } else {
      dma(lds, src, row_stride, valid);
    }
  }
  // MFMA fragment of row r for k-step ks, lane half `half`.
  template <typename M>
  __device__ static inline typename M::frag frag(const T* lds, int r, int ks, int half) {
    const char* base = reinterpret_cast<const char*>(lds);
    return M::load(reinterpret_cast<const T*>(base + off(r, ks * M::KSTEP + half * M::PER_LANE)));
  }
};

// The same 16-byte-per-lane global-to-LDS copy (to lds + 16 * lane) as
// inline assembly.  The compiler does not see an LDS store, so it adds no
// wait for the copy before later LDS reads (with the builtin it waits before
// any read it cannot prove disjoint, such as the other half of a
// double-buffered array); the caller orders every read of the destination
// after dma_wait() and a barrier.  Its own vector-memory waits stay correct:
// copies it does not count only make them stricter.  The copy takes its LDS
// address from M0, a register the compiler reserves and never treats as
// clobbered, so the statement saves M0 in a scratch SGPR of its own and
// restores it after issuing the copy (the copy reads M0 when it issues):
// whatever value the compiler keeps in M0 is unchanged across it.
__device__ inline void dma16_opaque(const void* g, void* lds) {
  const uint32_t m0 = (uint32_t)__builtin_amdgcn_readfirstlane(
      (int)(uintptr_t)(__attribute__((address_space(3))) void*)lds);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(g), "s"(m0)
      : "memory");
}

// dma16_opaque with the global address split into a wave-uniform base (in
// scalar registers) and a 32-bit per-lane byte offset, so that no 64-bit
// address arithmetic runs per lane.
__device__ inline void dma16_opaque_s(const void* base, uint32_t off, void* lds) {
  const uint32_t m0 = (uint32_t)__builtin_amdgcn_readfirstlane(
      (int)(uintptr_t)(__attribute__((address_space(3))) void*)lds);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off), "s"(base), "s"(m0)
      : "memory");
}

// A wave's DMA copies count as vector-memory loads; s_barrier does not wait
// for them on gfx950, so each wave drains its own copies before the barrier
// that hands the tile to the other waves.
__device__ inline void dma_wait() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// An empty asm statement that claims to rewrite `v`: later uses of `v` are
// ordered after it, and volatile statements keep their program order, so a
// sequence of pins fixes the order in which independent MFMA and VALU work
// is emitted.  It emits no instruction.
template <typename V>
__device__ inline void pin(V& v) { asm volatile("" : "+v"(v)); }


}  // namespace omnimem
