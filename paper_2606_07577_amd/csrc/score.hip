// Accumulated attention importance a_k (Eq. 6 of the OmniMem paper).
//
// a[g][j] sums, over every chunk query i of every query head h of KV head
// g, the softmax probability A[h][i][j] of the chunk attention (Eq. 1:
// one softmax over both caches and the visible chunk rows).  A row of A is
// only known once its normaliser is, so the work is two passes over the
// score matrix S = scale * Q K^T, both on MFMA tiles:
//   lse_pass     per (head, query, key range): running max and sum of
//                exp2 over the range (ranges split long rows over more
//                workgroups so that small layers still fill the chip)
//   colsum_pass  merges the range partials into the normaliser of each
//                query, then per (head, key): sum_i exp(S[i][j] - lse[i])
//   head_sum     a[g][j] = sum over the G query heads of KV head g.
// Scores stay in registers; nothing of size queries x keys touches HBM.
// Both passes stream one operand through double-buffered LDS (next tile
// prefetched into registers while the current one is consumed) and keep
// the other in registers, 64 rows per wavefront.  lse_merge joins them.
#include "common.h"

namespace omnimem {

namespace {

constexpr int kThreads = 256;       // 4 wavefronts
constexpr int kRowsPerWave = 64;    // register-resident rows per wave (two 32-wide MFMA blocks)
constexpr int kBlockRows = kScoreBlock;  // = 4 * kRowsPerWave
constexpr int kTile = kScoreTile;        // streamed rows per LDS stage
static_assert(kBlockRows == 4 * kRowsPerWave, "four waves per block");

__device__ inline float wave_xor32(float x) { return __shfl_xor(x, 32, 64); }

__device__ inline float max16(const floatx16& v) {
  float a = fmaxf(fmaxf(v[0], v[1]), v[2]);
  float b = fmaxf(fmaxf(v[3], v[4]), v[5]);
  float c = fmaxf(fmaxf(v[6], v[7]), v[8]);
  float d = fmaxf(fmaxf(v[9], v[10]), v[11]);
  float e = fmaxf(fmaxf(v[12], v[13]), v[14]);
  return fmaxf(fmaxf(fmaxf(a, b), fmaxf(c, d)), fmaxf(e, v[15]));
}


// Interleave `nm` MFMAs with the VALU work of the same basic block:
// groups of one MFMA followed by `nv` VALU instructions.
#define OMNIMEM_INTERLEAVE(nm, nv)                          \
  do {                                                      \
    _Pragma("unroll") for (int _i = 0; _i < (nm); ++_i) {   \
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);    \
      __builtin_amdgcn_sched_group_barrier(0x002, (nv), 0); \
    }                                                       \
  } while (0)

__device__ inline float max3f(float a, float b, float c) { return fmaxf(fmaxf(a, b), c); }

// Request the LDS fragments of one 32-row block for all k-steps.
template <typename M, typename Tl, int NKS, typename T>
__device__ inline void load_frags(typename M::frag (&f)[NKS], const T* lds, int row, int half) {
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) f[ks] = Tl::template frag<M>(lds, row, ks, half);
}

// 16 MFMAs: one 32-row block of an LDS stage against two 32-column blocks
// of register operands; each LDS fragment feeds two MFMAs.
template <typename M, typename Tile, int NKS, typename T>
__device__ inline void mma_rows(floatx16 (&acc)[2], const T* lds, int row, int half,
                                const typename M::frag (&b)[2][NKS]) {
  acc[0] = floatx16{};
  acc[1] = floatx16{};
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    const typename M::frag f = Tile::template frag<M>(lds, row, ks, half);
    acc[0] = M::mma(f, b[0][ks], acc[0]);
    acc[1] = M::mma(f, b[1][ks], acc[1]);
  }
}

// Running (max, sum) of exp2(sl2 * score) over the 16 scores of one query
// that a lane holds in an accumulator.
__device__ inline void online_update(const floatx16& acc, float sl2, float& m, float& lsum) {
  float mx = acc[0];
#pragma unroll
  for (int r = 1; r < 15; r += 2) mx = max3f(mx, acc[r], acc[r + 1]);
  mx = fmaxf(mx, acc[15]);
  const float mnew = fmaxf(m, mx * sl2);
  const float neg = -mnew;
  float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
  for (int r = 0; r < 16; r += 2) {
    s0 += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[r], sl2, neg));
    s1 += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[r + 1], sl2, neg));
  }
  lsum = lsum * __builtin_amdgcn_exp2f(m - mnew) + (s0 + s1);
  m = mnew;
}


// One pipeline phase of the LSE pass, scheduled by hand: the MFMAs of the
// 32-key row block `row` of an LDS stage (into `out`) alternate with the
// exp/sum work on the previous row block `in` (two query columns per lane,
// 16 scores each).  The work is software-pipelined across groups of one
// MFMA: a group issues its MFMA, the exps of scores whose exponents the
// previous group formed, the sums of the previous group's exps and the
// exponents of the next group, so no instruction waits on one issued just
// before it.
//
// Exponents are taken against the fixed reference m of the lane's query
// (not the block maximum), set by the caller from the segment's first keys:
// every exp2 stays finite while a score exceeds m by less than 2^7 in log2
// units, and sums up to ~2^100 lose nothing in fp32.  So the common path
// needs no maximum at all; the caller checks the sums at the segment's end.
//
// `f` holds the row block's LDS fragments, already requested.  With PF the
// phase also requests, spread over its groups, the fragments of row block
// `pf_row` of `pf_lds` into `pf` for the next phase.
template <typename M, typename Tl, bool PF, int NKS, typename T>
__device__ inline void lse_phase(floatx16 (&out)[2], typename M::frag (&f)[NKS], int half,
                                 typename M::frag (&qf)[2][NKS], const floatx16 (&in)[2], float sl2,
                                 float (&m)[2], float (&lsum)[2], const T* pf_lds, int pf_row,
                                 typename M::frag (&pf)[NKS]) {
  static_assert(16 % NKS == 0, "scores per k-step");
  constexpr int PER = 16 / NKS;   // scores of one column per group
  constexpr int NG = 2 * NKS;     // groups (one MFMA each)
  const float neg[2] = {-m[0], -m[1]};
  float y[2][PER], e[2][PER], s[2][2] = {{0.0f, 0.0f}, {0.0f, 0.0f}};
  // group g covers column cb = g & 1, scores (g >> 1) * PER .. + PER
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    y[0][i] = __builtin_fmaf(in[0][i], sl2, neg[0]);
    pin(y[0][i]);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int ks = g >> 1, cb = g & 1, b = g & 1;
    if (cb == 0) pin(f[ks]);
    pin(qf[cb][ks]);
    out[cb] = M::mma(f[ks], qf[cb][ks], ks ? out[cb] : floatx16{});
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      e[b][i] = __builtin_amdgcn_exp2f(y[b][i]);
      pin(e[b][i]);
    }
    if (g > 0) {
#pragma unroll
      for (int i = 0; i < PER; ++i) s[cb ^ 1][i & 1] += e[b ^ 1][i];
      pin(s[cb ^ 1][0]);
      pin(s[cb ^ 1][1]);
    }
    if (g + 1 < NG) {
      const int ncb = (g + 1) & 1, nks = (g + 1) >> 1;
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        y[b ^ 1][i] = __builtin_fmaf(in[ncb][nks * PER + i], sl2, neg[ncb]);
        pin(y[b ^ 1][i]);
      }
    }
    if (PF && cb == 1) pf[ks] = Tl::template frag<M>(pf_lds, pf_row, ks, half);
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int i = 0; i < PER; ++i) s[1][i & 1] += e[(NG - 1) & 1][i];
  lsum[0] += s[0][0] + s[0][1];
  lsum[1] += s[1][0] + s[1][1];
}

// Pass 1, one segment: for the 256 queries [q0, q0+256) of head h of layer
// l and the keys [kr0, kr1), the per-query reference m and sum of
// exp2(scale_log2 * q.k - m), merged over both lanes that share a query,
// written as partial `seg` of row `row`.
// MFMA tile: rows = 32 keys (A from LDS), columns = 32 queries (B in
// registers); each lane owns one query and 16 of its keys per tile.
// Software pipeline inside each wave: the MFMAs of one 32-key row block
// run while the exp/sum work of the previous row block executes; key tiles
// arrive by DMA one tile ahead into the LDS stage just consumed.
template <typename T, int D>
__device__ inline void lse_segment(const LayerDesc& Ld, const Dims& dm, int h, int q0, int kr0, int kr1,
                                   int64_t row, int seg, T* kt0, T* kt1, float2* __restrict__ part) {
  using M = Mfma<T>;
  using Tl = SwzTile<T, D>;
  constexpr int NKS = D / M::KSTEP;
  constexpr int NV = 2;                   // VALU per MFMA in the compiler-scheduled (fp32) path
  constexpr bool kHandSched = NKS <= 16;  // bf16: hand-interleaved phases
  const int C = Ld.n_chunk, N = Ld.n, nc = Ld.n_cache;

  const int wave = wave_id(), lane = threadIdx.x & 63, half = lane >> 5;
  const int g = h / dm.G;
  const T* q = reinterpret_cast<const T*>(Ld.q) + (int64_t)h * Ld.q_hs;
  const T* k = reinterpret_cast<const T*>(Ld.k) + (int64_t)g * Ld.kv_hs;
  const int64_t kv_rs = Ld.kv_rs;
  const int qw = q0 + wave * kRowsPerWave;
  const bool active = qw < C;
  const int kend_wave = min(kr1, dm.causal ? min(N, nc + min(qw + kRowsPerWave, C)) : N);

  // first tiles on their way before the query fragments are loaded
  const typename Tl::Plan plan = Tl::plan(kv_rs);
  Tl::copy(kt0, k + (int64_t)kr0 * kv_rs, kv_rs, min(kTile, N - kr0), plan);
  if (kr0 + kTile < kr1) Tl::copy(kt1, k + (int64_t)(kr0 + kTile) * kv_rs, kv_rs, min(kTile, N - kr0 - kTile), plan);

  typename M::frag qf[2][NKS];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    const int my_q = min(qw + cb * 32 + (lane & 31), C - 1);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      qf[cb][ks] = M::gload(q + (int64_t)my_q * Ld.q_rs + ks * M::KSTEP + half * M::PER_LANE);
  }
  const float sl2 = Ld.scale_log2;
  float m[2] = {-1e30f, -1e30f}, lsum[2] = {0.0f, 0.0f};

  // Scores of key row kb + off, off = acc_row(r) - half*4 (a constant), are
  // kept iff off <= lim; a 32-key row block needs masking only where it
  // passes the wave's key end or its first query's causal horizon.
  auto need_mask = [&](int kb) {
    return kb + 32 > kend_wave || (dm.causal && kb + 31 - nc > qw);
  };
  auto apply_mask = [&](floatx16 (&acc)[2], int kb) {
    const int base = kb + half * 4;
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
      int lim = kend_wave - 1 - base;
      if (dm.causal) lim = min(lim, qw + cb * 32 + (lane & 31) + nc - base);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int off = (r >> 2) * 8 + (r & 3);
        acc[cb][r] = off <= lim ? acc[cb][r] : -INFINITY;
      }
    }
  };

  const int arow = lane & 31;
  floatx16 acc0[2], acc1[2];  // [query column block] of key row block 0 / 1 of a tile
  typename M::frag fA[NKS], fB[NKS];  // LDS fragments of row block 1 / 0 of a tile
  dma_wait();
  __syncthreads();            // both first tiles landed in LDS for every wave
  if (active && kr0 < kend_wave) {
    mma_rows<M, Tl>(acc0, kt0, arow, half, qf);
    if constexpr (kHandSched) {
      load_frags<M, Tl>(fA, kt0, 32 + arow, half);
      // Reference of each query: the largest score among the segment's
      // first 32 keys.  A lane's visible keys form a prefix of the
      // segment's keys, so a lane with any visible key has one there.
      if (need_mask(kr0)) apply_mask(acc0, kr0);
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) {
        const float mx = fmaxf(max16(acc0[cb]), wave_xor32(max16(acc0[cb])));
        m[cb] = fmaxf(-1e30f, mx * sl2);
      }
    }
  }
  // One tile t in `cur`; tile t+1 is in (or on its way to) `nxt`.
  auto step = [&](int t, T* cur, const T* nxt) {
    const bool has_next = t + kTile < kr1;
    const bool busy = active && t < kend_wave;
    // phase A: MFMAs of key rows 32..63 of tile t || exp/sum of rows 0..31
    if (busy) {
      if (need_mask(t)) apply_mask(acc0, t);
      if constexpr (kHandSched) {
        lse_phase<M, Tl, false>(acc1, fA, half, qf, acc0, sl2, m, lsum, cur, 0, fB);
      } else {
        mma_rows<M, Tl>(acc1, cur, 32 + arow, half, qf);
        online_update(acc0[0], sl2, m[0], lsum[0]);
        online_update(acc0[1], sl2, m[1], lsum[1]);
        OMNIMEM_INTERLEAVE(16, NV);
      }
    }
    dma_wait();
    __syncthreads();  // tile t+1 landed; every wave is done with `cur`
    if (t + 2 * kTile < kr1)
      Tl::copy(cur, k + (int64_t)(t + 2 * kTile) * kv_rs, kv_rs, min(kTile, N - t - 2 * kTile), plan);
    // phase B: MFMAs of key rows 0..31 of tile t+1 || exp/sum of rows 32..63 of tile t
    if (busy) {
      if (need_mask(t + 32)) apply_mask(acc1, t + 32);
      if (has_next && t + kTile < kend_wave) {
        if constexpr (kHandSched) {
          load_frags<M, Tl>(fB, nxt, arow, half);
          lse_phase<M, Tl, true>(acc0, fB, half, qf, acc1, sl2, m, lsum, nxt, 32 + arow, fA);
        } else {
          mma_rows<M, Tl>(acc0, nxt, arow, half, qf);
          online_update(acc1[0], sl2, m[0], lsum[0]);
          online_update(acc1[1], sl2, m[1], lsum[1]);
          OMNIMEM_INTERLEAVE(16, NV);
        }
      } else {
        online_update(acc1[0], sl2, m[0], lsum[0]);
        online_update(acc1[1], sl2, m[1], lsum[1]);
      }
    }
  };
  for (int t = kr0; t < kr1; t += 2 * kTile) {
    step(t, kt0, kt1);
    if (t + kTile < kr1) step(t + kTile, kt1, kt0);
  }
  if constexpr (kHandSched) {
    // Later scores exceed the reference by far less than the sums' headroom
    // for any realistic input; a segment whose sums still leave it is redone
    // tile by tile with the reference moved to every block's maximum.
    const bool bad = active && !(lsum[0] < 0x1p100f && lsum[1] < 0x1p100f);
    if (__syncthreads_or(bad)) {  // also: every wave is done with the stages
      m[0] = m[1] = -1e30f;
      lsum[0] = lsum[1] = 0.0f;
      for (int t = kr0; t < kr1; t += kTile) {
        Tl::copy(kt0, k + (int64_t)t * kv_rs, kv_rs, min(kTile, N - t), plan);
        dma_wait();
        __syncthreads();
        if (active && t < kend_wave) {
#pragma unroll
          for (int rb = 0; rb < 2; ++rb) {
            mma_rows<M, Tl>(acc0, kt0, rb * 32 + arow, half, qf);
            if (need_mask(t + rb * 32)) apply_mask(acc0, t + rb * 32);
            online_update(acc0[0], sl2, m[0], lsum[0]);
            online_update(acc0[1], sl2, m[1], lsum[1]);
          }
        }
        __syncthreads();
      }
    }
  }
  if (!active) return;
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    const float m2 = wave_xor32(m[cb]), l2 = wave_xor32(lsum[cb]);
    const float mt = fmaxf(m[cb], m2);
    const float lt = lsum[cb] * __builtin_amdgcn_exp2f(m[cb] - mt) + l2 * __builtin_amdgcn_exp2f(m2 - mt);
    const int my_q = qw + cb * 32 + (lane & 31);
    if (half == 0 && my_q < C)
      part[(row * kMaxSeg + seg) * kBlockRows + (my_q - q0)] = make_float2(mt, lt);
  }
}

// Pass 1 over the plan's tiles (rows = (layer, head, 256-query block),
// tiles = the block's visible 64-key tiles): each workgroup walks its tile
// interval row by row.  Consecutive workgroups share rows and heads, so
// their logical ids go to one XCD's L2.
template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void lse_pass(const LayerDesc* __restrict__ layers, Dims dm, PassPlan pl,
                                                        float2* __restrict__ part) {
  using Tl = SwzTile<T, D>;
  __shared__ __attribute__((aligned(16))) T kt0[Tl::ELEMS];
  __shared__ __attribute__((aligned(16))) T kt1[Tl::ELEMS];
  const int i = gridDim.x % kXcds == 0 ? xcd_swizzle(blockIdx.x, gridDim.x) : (int)blockIdx.x;
  if (pl.c == 0) {  // row mode: row i, whole
    if (i >= pl.W) return;
    int l = 0;
    for (int lo = 0, hi = dm.L - 1; lo < hi;) {
      const int mid = (lo + hi + 1) >> 1;
      if (layers[mid].lse_rbase <= i) lo = mid; else hi = mid - 1;
      l = lo;
    }
    const LayerDesc Ld = layers[l];
    const int nb = (Ld.n_chunk + kBlockRows - 1) / kBlockRows;
    const int h = (int)((i - Ld.lse_rbase) / nb), b = (int)((i - Ld.lse_rbase) % nb);
    const int q0 = b * kBlockRows;
    const int kend_blk = dm.causal ? min(Ld.n, Ld.n_cache + min(q0 + kBlockRows, Ld.n_chunk)) : Ld.n;
    lse_segment<T, D>(Ld, dm, h, q0, 0, kend_blk, ((int64_t)l * dm.Hq + h) * dm.qb + b, 0, kt0, kt1, part);
    return;
  }
  bool first = true;
  for (int64_t chunk = i; chunk * pl.c < pl.W; chunk += pl.P) {
    int64_t g = chunk * pl.c;
    const int64_t gend = min(pl.W, g + pl.c);
    // the layer holding tile g: the last layer whose first tile is <= g
    int l = 0;
    for (int lo = 0, hi = dm.L - 1; lo < hi;) {
      const int mid = (lo + hi + 1) >> 1;
      if (layers[mid].lse_base <= g) lo = mid; else hi = mid - 1;
      l = lo;
    }
    LayerDesc Ld = layers[l];
    int h = (int)((g - Ld.lse_base) / Ld.lse_th);
    int ta = (int)((g - Ld.lse_base) % Ld.lse_th), b = 0;
    for (int t; ta >= (t = lse_row_tiles(Ld.n, Ld.n_cache, Ld.n_chunk, b, dm.causal)); ta -= t) ++b;
    for (; g < gend; first = false) {
      const int tiles = lse_row_tiles(Ld.n, Ld.n_cache, Ld.n_chunk, b, dm.causal);
      const int tb = (int)min((int64_t)tiles, ta + (gend - g));
      const int q0 = b * kBlockRows;
      const int kend_blk = dm.causal ? min(Ld.n, Ld.n_cache + min(q0 + kBlockRows, Ld.n_chunk)) : Ld.n;
      if (!first) __syncthreads();  // every wave is done with the stages of the previous segment
      lse_segment<T, D>(Ld, dm, h, q0, ta * kTile, min(tb * kTile, kend_blk),
                        ((int64_t)l * dm.Hq + h) * dm.qb + b, plan_seg(pl, g - ta, g), kt0, kt1, part);
      g += tb - ta;
      ta = 0;
      if (++b * kBlockRows >= Ld.n_chunk) {
        b = 0;
        if (++h == dm.Hq) {
          h = 0;
          do { ++l; } while (g < gend && l < dm.L && layers[l].lse_th == 0);
          if (g >= gend || l >= dm.L) break;
          Ld = layers[l];
        }
      }
    }
  }
}

// Normaliser of every chunk query in log2 units: the caller's lse, or the
// merge of the segment partials of the query's row (in segment order).
// Also writes the natural-log value to lse_out when requested.
__global__ __launch_bounds__(256) void lse_merge(const LayerDesc* __restrict__ layers, Dims dm, PassPlan pl,
                                                 const float2* __restrict__ part, float* __restrict__ lse2,
                                                 float* __restrict__ lse_out) {
  const int l = blockIdx.z, h = blockIdx.y;
  const LayerDesc Ld = layers[l];
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= Ld.n_chunk) return;
  const int64_t o = ((int64_t)l * dm.Hq + h) * dm.max_chunk + i;
  if (Ld.lse_in) {
    const float v = Ld.lse_in[(int64_t)h * Ld.n_chunk + i];
    lse2[o] = v * kLog2e;
    if (lse_out) lse_out[o] = v;
    return;
  }
  const int b = i / kBlockRows;
  int64_t start = Ld.lse_base + (int64_t)h * Ld.lse_th;
  for (int bb = 0; bb < b; ++bb) start += lse_row_tiles(Ld.n, Ld.n_cache, Ld.n_chunk, bb, dm.causal);
  const int tiles = lse_row_tiles(Ld.n, Ld.n_cache, Ld.n_chunk, b, dm.causal);
  const int nseg = plan_seg(pl, start, start + tiles - 1) + 1;
  const float2* p = part + ((((int64_t)l * dm.Hq + h) * dm.qb + b) * kMaxSeg) * kBlockRows + (i - b * kBlockRows);
  float2 v[kMaxSeg];  // all partials requested before the first is used
#pragma unroll
  for (int sg = 0; sg < kMaxSeg; ++sg) v[sg] = sg < nseg ? p[sg * kBlockRows] : make_float2(-1e30f, 0.0f);
  float mx = -1e30f, sum = 0.0f;
#pragma unroll
  for (int sg = 0; sg < kMaxSeg; ++sg) {
    const float m2 = fmaxf(mx, v[sg].x);
    sum = sum * __builtin_amdgcn_exp2f(mx - m2) + v[sg].y * __builtin_amdgcn_exp2f(v[sg].x - m2);
    mx = m2;
  }
  const float v2 = mx + __log2f(sum);
  lse2[o] = v2;
  if (lse_out) lse_out[o] = v2 * kLn2;
}

// cs[cb] += sum over the lane's 16 query rows of exp2(sl2 * score - lse2).
__device__ inline void colsum_update(const floatx16 (&acc)[2], const float* lse2_rows, int half, float sl2,
                                     float (&cs)[2]) {
  float nl[16];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const floatx4 v = *reinterpret_cast<const floatx4*>(lse2_rows + j * 8 + half * 4);
    nl[j * 4 + 0] = -v[0]; nl[j * 4 + 1] = -v[1]; nl[j * 4 + 2] = -v[2]; nl[j * 4 + 3] = -v[3];
  }
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; r += 2) {
      s0 += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[cb][r], sl2, nl[r]));
      s1 += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[cb][r + 1], sl2, nl[r + 1]));
    }
    cs[cb] += s0 + s1;
  }
}

// One pipeline phase of the column-sum pass, scheduled and software-
// pipelined like lse_phase: the MFMAs of query row block `row` (into `out`)
// alternate with exp2(score * sl2 - lse2) and its sum over the 16 query rows
// per lane of the previous row block `in`; row r's normaliser is
// lse2_rows[(r >> 2) * 8 + half * 4 + (r & 3)].
template <typename M, typename Tl, int NKS, typename T>
__device__ inline void colsum_phase(floatx16 (&out)[2], const T* lds, int row, int half,
                                    typename M::frag (&kf)[2][NKS], const floatx16 (&in)[2],
                                    const float* lse2_rows, float sl2, float (&cs)[2]) {
  static_assert(16 % NKS == 0, "scores per k-step");
  constexpr int PER = 16 / NKS;
  constexpr int NG = 2 * NKS;
  float nl[16];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const floatx4 v = *reinterpret_cast<const floatx4*>(lse2_rows + j * 8 + half * 4);
    nl[j * 4 + 0] = v[0]; nl[j * 4 + 1] = v[1]; nl[j * 4 + 2] = v[2]; nl[j * 4 + 3] = v[3];
  }
  typename M::frag f[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) f[ks] = Tl::template frag<M>(lds, row, ks, half);
  float y[2][PER], e[2][PER], s[2][2] = {{0.0f, 0.0f}, {0.0f, 0.0f}};
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    y[0][i] = __builtin_fmaf(in[0][i], sl2, -nl[i]);
    pin(y[0][i]);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int ks = g >> 1, cb = g & 1, b = g & 1;
    if (cb == 0) pin(f[ks]);
    pin(kf[cb][ks]);
    out[cb] = M::mma(f[ks], kf[cb][ks], ks ? out[cb] : floatx16{});
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      e[b][i] = __builtin_amdgcn_exp2f(y[b][i]);
      pin(e[b][i]);
    }
    if (g > 0) {
#pragma unroll
      for (int i = 0; i < PER; ++i) s[cb ^ 1][i & 1] += e[b ^ 1][i];
      pin(s[cb ^ 1][0]);
      pin(s[cb ^ 1][1]);
    }
    if (g + 1 < NG) {
      const int ncb = (g + 1) & 1, nks = (g + 1) >> 1;
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int r = nks * PER + i;
        y[b ^ 1][i] = __builtin_fmaf(in[ncb][r], sl2, -nl[r]);
        pin(y[b ^ 1][i]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int i = 0; i < PER; ++i) s[1][i & 1] += e[(NG - 1) & 1][i];
  cs[0] += s[0][0] + s[0][1];
  cs[1] += s[1][0] + s[1][1];
}

// Pass 2, one segment: per-query-head column sums sum_i exp(S[i][j] -
// lse[i]) for the 256 keys [k0, k0+256) of head h over the chunk queries
// [qstart, C), written as partial `seg` of row `row`.
// MFMA tile: rows = 32 queries (A from LDS), columns = 32 keys (B in
// registers, two blocks per wave); each lane accumulates one key's sum
// over 16 query rows per tile.  Software pipeline inside each wave: the
// MFMAs of one 32-query half run while the exp/sum work of the previous
// half executes; query tiles arrive by DMA one tile ahead.
template <typename T, int D>
__device__ inline void colsum_segment(const LayerDesc& Ld, const Dims& dm, int l, int h, int k0, int qstart,
                                      int C, int64_t row, int seg, T* qt0, T* qt1, float (&lse2)[3][kTile],
                                      const float* __restrict__ lse2_all, float* __restrict__ part) {
  using M = Mfma<T>;
  using Tl = SwzTile<T, D>;
  constexpr int NKS = D / M::KSTEP;
  constexpr int NV = 2;                   // VALU per MFMA in the compiler-scheduled (fp32) path
  constexpr bool kHandSched = NKS <= 16;  // bf16: hand-interleaved phases
  const int N = Ld.n, nc = Ld.n_cache;
  const int wave = wave_id(), lane = threadIdx.x & 63, half = lane >> 5;
  const int g = h / dm.G;
  const T* q = reinterpret_cast<const T*>(Ld.q) + (int64_t)h * Ld.q_hs;
  const T* k = reinterpret_cast<const T*>(Ld.k) + (int64_t)g * Ld.kv_hs;
  const int64_t q_rs = Ld.q_rs;
  const float* lse2_lh = lse2_all + ((int64_t)l * dm.Hq + h) * dm.max_chunk;
  const int kw = k0 + wave * kRowsPerWave;
  const bool active = kw < N;
  const int qfirst_wave = dm.causal ? max(0, kw - nc) : 0;
  // Normaliser of tile row threadIdx.x % 64, loaded unconditionally from an
  // index clamped into the slice; rows past it get +inf (probability 0)
  // where the value is stored.  (A conditional load into a register first
  // set to +inf would make the compiler wait for the tile copies issued
  // before it.)
  auto load_lse = [&](int qt) { return gload<float>(lse2_lh + min(qt + (int)(threadIdx.x & 63), C - 1)); };
  auto lse_or_inf = [&](int qt, float v) { return qt + (int)threadIdx.x < C ? v : INFINITY; };
  float lse_next = 0.0f;
  const typename Tl::Plan plan = Tl::plan(q_rs);
  if (qstart < C) {
    Tl::copy(qt0, q + (int64_t)qstart * q_rs, q_rs, min(kTile, C - qstart), plan);
    if (threadIdx.x < kTile) lse2[0][threadIdx.x] = lse_or_inf(qstart, load_lse(qstart));
    if (qstart + kTile < C) {
      Tl::copy(qt1, q + (int64_t)(qstart + kTile) * q_rs, q_rs, min(kTile, C - qstart - kTile), plan);
      lse_next = load_lse(qstart + kTile);
    }
  }

  typename M::frag kf[2][NKS];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    const int key = min(kw + cb * 32 + (lane & 31), N - 1);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      kf[cb][ks] = M::gload(k + (int64_t)key * Ld.kv_rs + ks * M::KSTEP + half * M::PER_LANE);
  }
  const float sl2 = Ld.scale_log2;
  float cs[2] = {0.0f, 0.0f};

  // Row block qb needs masking when a key of the wave lies past the causal
  // horizon of its first query; the score of (query qb + acc_row(r), key
  // kw + cb*32 + (lane & 31)) is kept iff (r >> 2) * 8 + (r & 3) >= dlim.
  auto need_mask = [&](int qb) { return dm.causal && kw + kRowsPerWave - 1 - nc > qb; };
  auto apply_mask = [&](floatx16 (&acc)[2], int qb) {
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) {
      const int dlim = kw + cb * 32 + (lane & 31) - nc - qb - half * 4;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[cb][r] = ((r >> 2) * 8 + (r & 3)) >= dlim ? acc[cb][r] : -INFINITY;
    }
  };

  if (qstart < C) {
    const int arow = lane & 31;
    floatx16 acc0[2], acc1[2];
    auto busy_at = [&](int qt) { return active && qt + kTile > qfirst_wave; };
    dma_wait();
    __syncthreads();  // first tiles landed in LDS for every wave
    if (busy_at(qstart)) mma_rows<M, Tl>(acc0, qt0, arow, half, kf);
    int slot = 0;
    // One tile in two halves: part_a (phase A and the store of the next
    // tile's normalisers) and part_b (the barrier, the next DMA, phase B).
    // The loop below starts each iteration with part_b, at the barrier that
    // waits for every copy anyway: at a loop header the compiler no longer
    // tells the two LDS stages apart and would make phase A wait for the
    // copy into the other stage.
    auto part_a = [&](int qt, T* cur) {
      const int next_slot = slot == 2 ? 0 : slot + 1;
      const bool has_next = qt + kTile < C;
      const bool busy = busy_at(qt);
      // phase A: MFMAs of row block 1 of tile qt || exp/sum of row block 0
      if (busy) {
        if (need_mask(qt)) apply_mask(acc0, qt);
        if constexpr (kHandSched) {
          colsum_phase<M, Tl>(acc1, cur, 32 + arow, half, kf, acc0, &lse2[slot][0], sl2, cs);
        } else {
          mma_rows<M, Tl>(acc1, cur, 32 + arow, half, kf);
          colsum_update(acc0, &lse2[slot][0], half, sl2, cs);
          OMNIMEM_INTERLEAVE(16, NV);
        }
      }
      if (has_next && threadIdx.x < kTile) lse2[next_slot][threadIdx.x] = lse_or_inf(qt + kTile, lse_next);
    };
    auto part_b = [&](int qt, T* cur, const T* nxt) {
      const int next_slot = slot == 2 ? 0 : slot + 1;
      const bool has_next = qt + kTile < C;
      const bool busy = busy_at(qt);
      dma_wait();
      __syncthreads();  // tile qt+1 landed; every wave is done with `cur`
      if (qt + 2 * kTile < C) {
        Tl::copy(cur, q + (int64_t)(qt + 2 * kTile) * q_rs, q_rs, min(kTile, C - qt - 2 * kTile), plan);
        lse_next = load_lse(qt + 2 * kTile);
      }
      // phase B: MFMAs of row block 0 of tile qt+1 || exp/sum of row block 1.
      // A wave's tiles go from idle to busy (causal), so the next tile's
      // first MFMAs are issued whether or not this tile was busy.
      const bool busy_next = has_next && busy_at(qt + kTile);
      if (busy && need_mask(qt + 32)) apply_mask(acc1, qt + 32);
      if (busy && busy_next) {
        if constexpr (kHandSched) {
          colsum_phase<M, Tl>(acc0, nxt, arow, half, kf, acc1, &lse2[slot][32], sl2, cs);
        } else {
          mma_rows<M, Tl>(acc0, nxt, arow, half, kf);
          colsum_update(acc1, &lse2[slot][32], half, sl2, cs);
          OMNIMEM_INTERLEAVE(16, NV);
        }
      } else if (busy) {
        colsum_update(acc1, &lse2[slot][32], half, sl2, cs);
      } else if (busy_next) {
        mma_rows<M, Tl>(acc0, nxt, arow, half, kf);
      }
      slot = next_slot;
    };
    part_a(qstart, qt0);
    for (int qt = qstart;; qt += 2 * kTile) {
      part_b(qt, qt0, qt1);
      if (qt + kTile >= C) break;
      part_a(qt + kTile, qt1);
      part_b(qt + kTile, qt1, qt0);
      if (qt + 2 * kTile >= C) break;
      part_a(qt + 2 * kTile, qt0);
    }
  }
  if (!active) return;
  cs[0] += wave_xor32(cs[0]);
  cs[1] += wave_xor32(cs[1]);
  const int key = kw + half * 32 + (lane & 31);
  if (key < N) part[(row * kMaxSeg + seg) * kBlockRows + (key - k0)] = half ? cs[1] : cs[0];
}

// Pass 2 over the plan's tiles (rows = (layer, head, 256-key block), tiles
// = the 64-query tiles that see a key of the block), walked like lse_pass.
template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void colsum_pass(const LayerDesc* __restrict__ layers, Dims dm,
                                                           PassPlan pl, const float* __restrict__ lse2_all,
                                                           float* __restrict__ part) {
  using Tl = SwzTile<T, D>;
  __shared__ __attribute__((aligned(16))) T qt0[Tl::ELEMS];
  __shared__ __attribute__((aligned(16))) T qt1[Tl::ELEMS];
  // normalisers: three slots, because phase B of tile i still reads slot i
  // while a faster wave already stores tile i + 2's values
  __shared__ __attribute__((aligned(16))) float lse2[3][kTile];
  const int i = gridDim.x % kXcds == 0 ? xcd_swizzle(blockIdx.x, gridDim.x) : (int)blockIdx.x;
  if (pl.c == 0) {  // row mode: row i, whole
    if (i >= pl.W) return;
    int l = 0;
    for (int lo = 0, hi = dm.L - 1; lo < hi;) {
      const int mid = (lo + hi + 1) >> 1;
      if (layers[mid].cs_rbase <= i) lo = mid; else hi = mid - 1;
      l = lo;
    }
    const LayerDesc Ld = layers[l];
    const int nb = (Ld.n + kBlockRows - 1) / kBlockRows;
    const int h = (int)((i - Ld.cs_rbase) / nb), b = (int)((i - Ld.cs_rbase) % nb);
    const int t0 = cs_first_tile(Ld.n_cache, b, dm.causal);
    colsum_segment<T, D>(Ld, dm, l, h, b * kBlockRows, t0 * kTile, Ld.n_chunk, ((int64_t)l * dm.Hq + h) * dm.kb + b, 0,
                         qt0, qt1, lse2, lse2_all, part);
    return;
  }
  bool first = true;
  for (int64_t chunk = i; chunk * pl.c < pl.W; chunk += pl.P) {
    int64_t g = chunk * pl.c;
    const int64_t gend = min(pl.W, g + pl.c);
    int l = 0;
    for (int lo = 0, hi = dm.L - 1; lo < hi;) {
      const int mid = (lo + hi + 1) >> 1;
      if (layers[mid].cs_base <= g) lo = mid; else hi = mid - 1;
      l = lo;
    }
    LayerDesc Ld = layers[l];
    int h = (int)((g - Ld.cs_base) / Ld.cs_th);
    int ta = (int)((g - Ld.cs_base) % Ld.cs_th), b = 0;
    for (int t; ta >= (t = cs_row_tiles(Ld.n, Ld.n_cache, Ld.n_chunk, b, dm.causal)); ta -= t) ++b;
    for (; g < gend; first = false) {
      const int tiles = cs_row_tiles(Ld.n, Ld.n_cache, Ld.n_chunk, b, dm.causal);
      const int tb = (int)min((int64_t)tiles, ta + (gend - g));
      const int t0 = cs_first_tile(Ld.n_cache, b, dm.causal);
      if (!first) __syncthreads();  // every wave is done with the stages of the previous segment
      colsum_segment<T, D>(Ld, dm, l, h, b * kBlockRows, (t0 + ta) * kTile, min(Ld.n_chunk, (t0 + tb) * kTile),
                           ((int64_t)l * dm.Hq + h) * dm.kb + b, plan_seg(pl, g - ta, g), qt0, qt1, lse2,
                           lse2_all, part);
      g += tb - ta;
      ta = 0;
      if (++b * kBlockRows >= Ld.n) {
        b = 0;
        if (++h == dm.Hq) {
          h = 0;
          do { ++l; } while (g < gend && l < dm.L && layers[l].cs_th == 0);
          if (g >= gend || l >= dm.L) break;
          Ld = layers[l];
        }
      }
    }
  }
}

// a[l][g][j] = sum over the G query heads of KV head g and the segments of
// their column-sum rows, in a fixed order.
__global__ void head_sum(const LayerDesc* __restrict__ layers, Dims dm, PassPlan pl,
                         const float* __restrict__ part, float* __restrict__ a) {
  const int l = blockIdx.z, g = blockIdx.y;
  const LayerDesc Ld = layers[l];
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= Ld.n) return;
  const int b = j / kBlockRows;
  float sum = 0.0f;
  const int tiles = cs_row_tiles(Ld.n, Ld.n_cache, Ld.n_chunk, b, dm.causal);
  if (Ld.cs_th > 0 && tiles > 0) {
    int64_t start = Ld.cs_base;
    for (int bb = 0; bb < b; ++bb) start += cs_row_tiles(Ld.n, Ld.n_cache, Ld.n_chunk, bb, dm.causal);
    // the segment partials of up to kHeadsAtOnce query heads requested at
    // once, then added in head and segment order
    constexpr int kHeadsAtOnce = 8;
    for (int h0 = 0; h0 < dm.G; h0 += kHeadsAtOnce) {
      float v[kHeadsAtOnce][kMaxSeg];
#pragma unroll
      for (int u = 0; u < kHeadsAtOnce; ++u) {
        const int h = g * dm.G + min(h0 + u, dm.G - 1);  // (heads past G load nothing)
        const int64_t s0 = start + (int64_t)h * Ld.cs_th;
        const int nseg = h0 + u < dm.G ? plan_seg(pl, s0, s0 + tiles - 1) + 1 : 0;
        const float* p =
            part + ((((int64_t)l * dm.Hq + h) * dm.kb + b) * kMaxSeg) * kBlockRows + (j - b * kBlockRows);
#pragma unroll
        for (int sg = 0; sg < kMaxSeg; ++sg) v[u][sg] = sg < nseg ? p[sg * kBlockRows] : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < kHeadsAtOnce; ++u)
#pragma unroll
        for (int sg = 0; sg < kMaxSeg; ++sg) sum += v[u][sg];
    }
  }
  a[((int64_t)l * dm.Hkv + g) * dm.max_tokens + j] = sum;
}

template <typename T, int D>
void launch_typed(const Dims& dm, const LayerDesc* desc, const Workspace& ws, const PassPlan& lp,
                  const PassPlan& cp, float* lse_out, float* a, hipStream_t st) {
  if (lp.W > 0)
    OMNIMEM_LAUNCH(ws, K_LSE, st, lse_pass<T, D><<<lp.P, kThreads, 0, st>>>(desc, dm, lp, ws.lse_part));
  dim3 gm((unsigned)((dm.max_chunk + 255) / 256), dm.Hq, dm.L);
  OMNIMEM_LAUNCH(ws, K_LSE_MERGE, st, lse_merge<<<gm, 256, 0, st>>>(desc, dm, lp, ws.lse_part, ws.lse2, lse_out));
  if (cp.W > 0)
    OMNIMEM_LAUNCH(ws, K_COLSUM, st, colsum_pass<T, D><<<cp.P, kThreads, 0, st>>>(desc, dm, cp, ws.lse2, ws.part));
  dim3 g3((unsigned)((dm.max_tokens + 255) / 256), dm.Hkv, dm.L);
  OMNIMEM_LAUNCH(ws, K_HEADSUM, st, head_sum<<<g3, 256, 0, st>>>(desc, dm, cp, ws.part, a));
}

// Plan a pass of W tiles in `rows` rows, the longest of t_max tiles.  With
// rows to spare (at least 8 per workgroup slot) the hardware dispatcher
// balances one workgroup per row best.  Otherwise chunks hold at least
// t_max / (kMaxSeg - 1) tiles (the bound on segments per row) and, if the
// work allows, about two rows (a segment's start costs about as much as a
// few tiles); then as many rounds of P chunks as fit, with the chunk size
// that fills the rounds evenly.
PassPlan choose_plan(int64_t W, int64_t rows, int t_max, int max_workgroups) {
  PassPlan p{W, 0, 1};
  if (W <= 0) return p;
  if (rows >= 8 * (int64_t)max_workgroups && rows < (int64_t{1} << 31) / 2) {
    p.W = rows;
    p.P = (int)xcd_grid(rows);
    p.c = 0;
    return p;
  }
  const int64_t c_min = std::max<int64_t>((t_max + kMaxSeg - 2) / (kMaxSeg - 1), 1);
  const int64_t c_pref = std::max<int64_t>(c_min, std::max(2 * t_max, 32));
  if (W <= (int64_t)max_workgroups * c_pref) {
    p.P = (int)std::max<int64_t>(1, std::min<int64_t>(max_workgroups, W / c_min));
    if (p.P >= kXcds) p.P = p.P / kXcds * kXcds;
    p.c = (int)((W + p.P - 1) / p.P);
  } else {
    const int64_t rounds = W / ((int64_t)max_workgroups * c_pref);
    p.c = (int)((W + (int64_t)max_workgroups * rounds - 1) / ((int64_t)max_workgroups * rounds));
    p.P = max_workgroups / kXcds * kXcds;
  }
  return p;
}

}  // namespace

// Fill each layer's tile bases of both score passes and the two plans.
void plan_score(const Dims& dm, LayerDesc* layers, int max_workgroups, PassPlan* lse_plan, PassPlan* cs_plan) {
  int64_t lse_w = 0, cs_w = 0, lse_rows = 0, cs_rows = 0;
  int lse_tmax = 0, cs_tmax = 0;
  for (int l = 0; l < dm.L; ++l) {
    LayerDesc& x = layers[l];
    int th = 0, nb = 0;
    if (!x.lse_in) {
      for (int b = 0; b * kBlockRows < x.n_chunk; ++b, ++nb) {
        const int t = lse_row_tiles(x.n, x.n_cache, x.n_chunk, b, dm.causal);
        th += t;
        lse_tmax = std::max(lse_tmax, t);
      }
    }
    x.lse_base = lse_w;
    x.lse_th = th;
    x.lse_rbase = lse_rows;
    lse_w += (int64_t)dm.Hq * th;
    lse_rows += th > 0 ? (int64_t)dm.Hq * nb : 0;
    int ch = 0;
    nb = 0;
    for (int b = 0; b * kBlockRows < x.n; ++b, ++nb) {
      const int t = cs_row_tiles(x.n, x.n_cache, x.n_chunk, b, dm.causal);
      ch += t;
      cs_tmax = std::max(cs_tmax, t);
    }
    x.cs_base = cs_w;
    x.cs_th = ch;
    x.cs_rbase = cs_rows;
    cs_w += (int64_t)dm.Hq * ch;
    cs_rows += ch > 0 ? (int64_t)dm.Hq * nb : 0;
  }
  *lse_plan = choose_plan(lse_w, lse_rows, lse_tmax, max_workgroups);
  *cs_plan = choose_plan(cs_w, cs_rows, cs_tmax, max_workgroups);
}

hipError_t launch_score(const Dims& dm, int dtype, const LayerDesc* desc, const Workspace& ws,
                        const PassPlan& lse_plan, const PassPlan& cs_plan, float* lse_out, float* a,
                        hipStream_t st) {
  if (dtype == 0) {
    if (dm.d == 128) launch_typed<uint16_t, 128>(dm, desc, ws, lse_plan, cs_plan, lse_out, a, st);
    else launch_typed<uint16_t, 64>(dm, desc, ws, lse_plan, cs_plan, lse_out, a, st);
  } else {
    if (dm.d == 128) launch_typed<float, 128>(dm, desc, ws, lse_plan, cs_plan, lse_out, a, st);
    else launch_typed<float, 64>(dm, desc, ws, lse_plan, cs_plan, lse_out, a, st);
  }
  return hipGetLastError();
}

}  // namespace omnimem
