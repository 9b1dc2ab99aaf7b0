// Cosine-similarity redundancy s_k (Eq. 7 of the OmniMem paper, computed
// from value vectors as Sec. 3.1 allows, or keys).
//
// Two modes:
//  SIM_MAX  s_k = max over the other rows j of k's (KV head, modality)
//           segment of cos(u_k, u_j).  The segment's Gram matrix U U^T is
//           tiled 128 x 128 over its upper triangle on MFMA (raw bf16/fp32
//           inputs, fp32 accumulation), scaled by fp32 inverse norms, and
//           reduced to row and column maxima in registers; maxima merge with
//           atomicMax on an order-preserving int encoding.  The N x N matrix
//           never leaves the chip.
//  SIM_ADJ  Eq. (7) as printed: mean cosine with the previous and next row
//           of the same modality, in fp64.
#include "common.h"

namespace omnimem {

namespace {

// --- modality lists --------------------------------------------------------
// Per layer: pos[l][0][0 .. K_v) = visual rows ascending, pos[l][1][0 .. K_a)
// = audio rows ascending; rank[j] = index of row j inside its modality's
// list.  One pass, 16 rows per thread.
constexpr int kListPer = 16;

__device__ inline int64_t plan_F(int64_t n);

__global__ __launch_bounds__(1024) void modality_lists(const LayerDesc* __restrict__ layers, Dims dm,
                                                      int* __restrict__ pos, int* __restrict__ rank,
                                                      int* __restrict__ counts, int4* __restrict__ items,
                                                      int* __restrict__ n_items, int64_t items_per_layer,
                                                      int make_plan) {
  const int l = blockIdx.x;
  const int N = layers[l].n;
  const uint8_t* mod = layers[l].mod;
  __shared__ int wave_tot[16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwaves = blockDim.x >> 6;
  int* Pv = pos + (int64_t)(2 * l) * dm.max_tokens;
  int* Pa = Pv + dm.max_tokens;
  int* R = rank + (int64_t)l * dm.max_tokens;
  int carry = 0;  // visual rows before the current span
  for (int base = 0; base < N; base += (int)blockDim.x * kListPer) {
    const int j0 = base + (int)threadIdx.x * kListPer;
    uint8_t m[kListPer];
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < kListPer; ++e) {
      m[e] = j0 + e < N ? mod[j0 + e] : 1;
      cnt += m[e] == 0;
    }
    int incl = cnt;  // inclusive scan over the wave
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(incl, o, 64);
      if (lane >= o) incl += t;
    }
    __syncthreads();
    if (lane == 63) wave_tot[wave] = incl;
    __syncthreads();
    int rv = carry + incl - cnt, span = 0;
    for (int w = 0; w < nwaves; ++w) {
      rv += w < wave ? wave_tot[w] : 0;
      span += wave_tot[w];
    }
#pragma unroll
    for (int e = 0; e < kListPer; ++e) {
      const int j = j0 + e;
      if (j >= N) break;
      if (m[e] == 0) { Pv[rv] = j; R[j] = rv; ++rv; }
      else { const int ra = j - rv; Pa[ra] = j; R[j] = ra; }
    }
    carry += span;
  }
  const int kv = carry;
  if (threadIdx.x == 0) { counts[2 * l] = kv; counts[2 * l + 1] = N - kv; }
  if (!make_plan) return;

  // Gram work plan of this layer, in its own slot range [l * per_layer, ...):
  // segment (g, mu) with T = ceil(K / 128) row blocks owns, for row block
  // I, ceil((T - I) / S) items of up to S column blocks.
  __syncthreads();
  int4* it = items + (int64_t)l * items_per_layer;
  int64_t ibase = 0;
  for (int g = 0; g < dm.Hkv; ++g)
    for (int smu = 0; smu < 2; ++smu) {
      const int K = smu ? N - kv : kv;
      const int T = (K + kGramTile - 1) / kGramTile;
      const int64_t FT = plan_F(T);
      const int seg = (l * dm.Hkv + g) * 2 + smu;
      for (int I = threadIdx.x; I < T; I += blockDim.x) {
        int64_t o = ibase + FT - plan_F(T - I);
        for (int J0 = I; J0 < T; J0 += kGramStrip, ++o)
          if (o < items_per_layer) it[o] = make_int4(seg, I, J0, min(T, J0 + kGramStrip));
      }
      ibase += FT;
    }
  if (threadIdx.x == 0) n_items[l] = (int)min<int64_t>(ibase, items_per_layer);
}

// --- Gram work plan ----------------------------------------------------------
// Segment (l, g, mu) with T = ceil(K / 128) row blocks owns, for each row
// block I, ceil((T - I) / S) items covering column blocks [J0, J0 + S).
// F(n) = sum_{m=1..n} ceil(m / S) counts the items of rows with n blocks.
__device__ inline int64_t plan_F(int64_t n) {
  const int64_t q = n / kGramStrip, r = n % kGramStrip;
  return kGramStrip * q * (q + 1) / 2 + r * (q + 1);
}

// --- inverse norms -----------------------------------------------------------
// inv_norm[l][g][j] = 1 / ||u_j|| (0 for a zero row), accumulated in fp64.
template <typename T, int D>
__global__ __launch_bounds__(256) void inv_norms(const LayerDesc* __restrict__ layers, Dims dm, int on_keys,
                                                 float* __restrict__ inv, int* __restrict__ best) {
  const int l = blockIdx.z, g = blockIdx.y;
  const LayerDesc Ld = layers[l];
  const int N = Ld.n;
  constexpr int LPR = 16;                              // lanes per row
  constexpr int EPL = D / LPR;                         // elements per lane
  const int row = blockIdx.x * (256 / LPR) + threadIdx.x / LPR;
  const int sub = threadIdx.x % LPR;
  const T* u = reinterpret_cast<const T*>(on_keys ? Ld.k : Ld.v) + (int64_t)g * Ld.kv_hs;
  double acc = 0.0;
  if (row < N) {
    const T* p = u + (int64_t)row * Ld.kv_rs + sub * EPL;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      float x;
      if constexpr (sizeof(T) == 2) x = __uint_as_float(((uint32_t)p[e]) << 16);
      else x = p[e];
      acc += (double)x * (double)x;
    }
  }
#pragma unroll
  for (int o = LPR / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
  if (row < N && sub == 0) {
    const int64_t o = ((int64_t)l * dm.Hkv + g) * dm.max_tokens + row;
    inv[o] = acc > 0.0 ? (float)(1.0 / sqrt(acc)) : 0.0f;
    best[o] = kNoPartner;  // the Gram pass merges maxima into this
  }
}


// --- Gram max -------------------------------------------------------------
// One work item = row block I (128 rows) of a segment against column blocks
// [J0, J1).  Wave w keeps rows w*32 .. w*32+31 of block I as MFMA A operands
// in registers for the whole item and streams each 128-row column block
// through double-buffered LDS (B operands, 4 column tiles of 32).  Per
// element: cos = dot * inv_i * inv_j.  Column maxima are reduced in
// registers per tile and merged with atomicMax at once; row maxima are
// carried across the strip and reduced across lanes at the end.  Rows and
// columns past the segment get a NaN inverse norm, which fmaxf ignores.
template <typename T, int D>
struct GramStage {
  static constexpr int CPR = D * (int)sizeof(T) / 16;
  static constexpr int PER_THREAD = kGramTile * CPR / 256;
  static constexpr int LD = D + lds_pad<T>();
  uint4 r[PER_THREAD];
  // rows `rows_idx[0 .. valid)` of u; the rest repeat row rows_idx[valid - 1]
  __device__ inline void load(const T* u, int64_t row_stride, const int* rows_idx, int valid) {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = threadIdx.x + i * 256;
      const int row = c / CPR, x = c % CPR;
      const int src = rows_idx[min(row, valid - 1)];
      r[i] = gload16(u + (int64_t)src * row_stride + x * (16 / sizeof(T)));
    }
  }
  __device__ inline void store(T* lds) const {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = threadIdx.x + i * 256;
      const int row = c / CPR, x = c % CPR;
      *reinterpret_cast<uint4*>(lds + row * LD + x * (16 / sizeof(T))) = r[i];
    }
  }
};

// Accumulator register r holds tile row (r >> 2) * 8 + half * 4 + (r & 3):
// it is the lane's own column when (r >> 2) * 8 + (r & 3) == d.
__device__ inline void drop_diagonal(floatx16& a, int d) {
#pragma unroll
  for (int r = 0; r < 16; ++r) a[r] = ((r >> 2) * 8 + (r & 3)) == d ? __builtin_nanf("") : a[r];
}

template <typename T, int D>
__global__ __launch_bounds__(256, 2) void gram_max(const LayerDesc* __restrict__ layers, Dims dm, int on_keys,
                                                   const int* __restrict__ pos, const int* __restrict__ counts,
                                                   const float* __restrict__ inv, const int4* __restrict__ items,
                                                   const int* __restrict__ n_items, int64_t items_per_layer,
                                                   int* __restrict__ best) {
  using M = Mfma<T>;
  using S = GramStage<T, D>;
  constexpr int NKS = D / M::KSTEP;
  constexpr int LD = S::LD;
  constexpr int TB = kGramTile;
  __shared__ __attribute__((aligned(16))) T tJ[2][TB * LD];
  __shared__ float invJ[2][TB];
  __shared__ int rowsJ[2][TB];

  const int wave = wave_id(), lane = threadIdx.x & 63, half = lane >> 5;
  const int64_t total = (int64_t)dm.L * items_per_layer;

  for (int64_t it = blockIdx.x; it < total; it += gridDim.x) {
    if (it % items_per_layer >= n_items[it / items_per_layer]) continue;  // unused slot
    const int4 item = items[it];
    const int seg = item.x, I = item.y, J0 = item.z, J1 = item.w;
    const int l = seg / (dm.Hkv * 2), g = (seg >> 1) % dm.Hkv, mu = seg & 1;
    const int K = counts[2 * l + mu];
    const int* P = pos + (int64_t)(2 * l + mu) * dm.max_tokens;
    const int64_t kv_rs = layers[l].kv_rs;
    const T* u = reinterpret_cast<const T*>(on_keys ? layers[l].k : layers[l].v) + (int64_t)g * layers[l].kv_hs;
    const float* inv_g = inv + ((int64_t)l * dm.Hkv + g) * dm.max_tokens;
    int* best_g = best + ((int64_t)l * dm.Hkv + g) * dm.max_tokens;

    // this wave's 32 rows of block I: A fragments and inverse norms
    const int validI = min(TB, K - I * TB);
    const int r0 = wave * 32;
    const bool wave_rows = r0 < validI;
    const int my_row = r0 + (lane & 31);
    const int my_pos = P[I * TB + min(my_row, validI - 1)];
    typename M::frag af[NKS];
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      af[ks] = M::gload(u + (int64_t)my_pos * kv_rs + ks * M::KSTEP + half * M::PER_LANE);
    float ri[16];  // inverse norms of the 16 rows this lane's accumulators hold
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = r0 + acc_row(r, lane);
      ri[r] = row < validI ? inv_g[P[I * TB + row]] : __builtin_nanf("");
    }
    float rmax[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) rmax[r] = -INFINITY;

    S pre;
    __syncthreads();  // the previous item is done with the LDS buffers
    {
      const int validJ = min(TB, K - J0 * TB);
      if (threadIdx.x < TB) {
        const int c = threadIdx.x;
        const int p = P[J0 * TB + min(c, validJ - 1)];
        rowsJ[0][c] = p;
        invJ[0][c] = c < validJ ? inv_g[p] : __builtin_nanf("");
      }
      __syncthreads();
      pre.load(u, kv_rs, rowsJ[0], validJ);
      pre.store(tJ[0]);
    }
    int buf = 0;
    for (int J = J0; J < J1; ++J, buf ^= 1) {
      const bool has_next = J + 1 < J1;
      int validJn = 0;
      if (has_next) {
        validJn = min(TB, K - (J + 1) * TB);
        if (threadIdx.x < TB) {
          const int c = threadIdx.x;
          const int p = P[(J + 1) * TB + min(c, validJn - 1)];
          rowsJ[buf ^ 1][c] = p;
          invJ[buf ^ 1][c] = c < validJn ? inv_g[p] : __builtin_nanf("");
        }
      }
      __syncthreads();  // tJ[buf] staged; rowsJ[buf ^ 1] written
      if (has_next) pre.load(u, kv_rs, rowsJ[buf ^ 1], validJn);
      const int validJ = min(TB, K - J * TB);
      if (wave_rows) {
        floatx16 acc[4];
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) acc[ct] = floatx16{};
        const T* b0 = tJ[buf] + (lane & 31) * LD + half * M::PER_LANE;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
          for (int ct = 0; ct < 4; ++ct)
            acc[ct] = M::mma(af[ks], M::load(b0 + ct * 32 * LD + ks * M::KSTEP), acc[ct]);
        if (I == J) {
          // the pair (row, row) lies in column tile `wave`: drop it
          const int d = (lane & 31) - half * 4;
          switch (wave) {
            case 0: drop_diagonal(acc[0], d); break;
            case 1: drop_diagonal(acc[1], d); break;
            case 2: drop_diagonal(acc[2], d); break;
            default: drop_diagonal(acc[3], d); break;
          }
        }
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) {
          const int cj = ct * 32 + (lane & 31);
          const float ij = invJ[buf][cj];
          float cm = -INFINITY;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            cm = fmaxf(cm, acc[ct][r] * ri[r]);
            rmax[r] = fmaxf(rmax[r], acc[ct][r] * ij);
          }
          // both row halves of column cj, scaled by its inverse norm
          cm = fmaxf(cm, __shfl_xor(cm, 32, 64));
          if (half == 0 && cj < validJ && cm > -INFINITY) {
            const float c = fminf(1.0f, fmaxf(-1.0f, cm * ij));
            atomicMax(best_g + rowsJ[buf][cj], ord_f32(c));
          }
        }
      }
      if (has_next) pre.store(tJ[buf ^ 1]);
    }
    // Row maxima: reduce over the 32 lanes of each half, then merge.
    if (wave_rows) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v = rmax[r];
#pragma unroll
        for (int o = 16; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
        rmax[r] = v;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = r0 + acc_row(r, lane);
        if ((lane & 31) == r && row < validI && rmax[r] > -INFINITY) {
          const float c = fminf(1.0f, fmaxf(-1.0f, rmax[r] * ri[r]));
          atomicMax(best_g + P[I * TB + row], ord_f32(c));
        }
      }
    }
  }
}

// s[l][g][j] from the merged maxima; a row with no partner gets 0.
__global__ void gram_finish(const LayerDesc* __restrict__ layers, Dims dm, const int* __restrict__ best,
                            float* __restrict__ s) {
  const int l = blockIdx.z, g = blockIdx.y;
  const int N = layers[l].n;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= N) return;
  const int64_t o = ((int64_t)l * dm.Hkv + g) * dm.max_tokens + j;
  const int b = best[o];
  s[o] = b == kNoPartner ? 0.0f : fminf(1.0f, fmaxf(-1.0f, unord_f32(b)));
}

// --- SIM_ADJ: Eq. (7) with the modality's own neighbours --------------------
template <typename T, int D>
__device__ double cos64(const T* x, const T* y) {
  double xy = 0.0, xx = 0.0, yy = 0.0;
  for (int e = 0; e < D; ++e) {
    double a, b;
    if constexpr (sizeof(T) == 2) { a = __uint_as_float(((uint32_t)x[e]) << 16); b = __uint_as_float(((uint32_t)y[e]) << 16); }
    else { a = x[e]; b = y[e]; }
    xy += a * b; xx += a * a; yy += b * b;
  }
  if (xx <= 0.0 || yy <= 0.0) return 0.0;
  const double c = xy / (sqrt(xx) * sqrt(yy));
  return c > 1.0 ? 1.0 : (c < -1.0 ? -1.0 : c);
}

template <typename T, int D>
__global__ void adjacent_cos(const LayerDesc* __restrict__ layers, Dims dm, int on_keys, const int* __restrict__ pos,
                             const int* __restrict__ rank, const int* __restrict__ counts, float* __restrict__ s) {
  const int l = blockIdx.z, g = blockIdx.y;
  const LayerDesc Ld = layers[l];
  const int N = Ld.n;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= N) return;
  const int mu = Ld.mod[j] ? 1 : 0;
  const int K = counts[2 * l + mu];
  const int* P = pos + (int64_t)(2 * l + mu) * dm.max_tokens;
  const int t = rank[(int64_t)l * dm.max_tokens + j];
  const T* u = reinterpret_cast<const T*>(on_keys ? Ld.k : Ld.v) + (int64_t)g * Ld.kv_hs;
  const T* x = u + (int64_t)j * Ld.kv_rs;
  double sum = 0.0;
  int n = 0;
  if (t > 0) { sum += cos64<T, D>(x, u + (int64_t)P[t - 1] * Ld.kv_rs); ++n; }
  if (t + 1 < K) { sum += cos64<T, D>(x, u + (int64_t)P[t + 1] * Ld.kv_rs); ++n; }
  s[((int64_t)l * dm.Hkv + g) * dm.max_tokens + j] = n ? (float)(sum / n) : 0.0f;
}

template <typename T, int D>
void launch_typed(const Dims& dm, int sim, int on_keys, const LayerDesc* desc, const Workspace& ws, float* s,
                  hipStream_t st) {
  const dim3 gtok((unsigned)((dm.max_tokens + 255) / 256), dm.Hkv, dm.L);
  if (sim == 1) {
    OMNIMEM_LAUNCH(ws, K_ADJ, st, adjacent_cos<T, D><<<gtok, 256, 0, st>>>(desc, dm, on_keys, ws.pos, ws.rank, ws.counts, s));
    return;
  }
  const dim3 gnorm((unsigned)((dm.max_tokens + 15) / 16), dm.Hkv, dm.L);
  OMNIMEM_LAUNCH(ws, K_NORMS, st, inv_norms<T, D><<<gnorm, 256, 0, st>>>(desc, dm, on_keys, ws.inv_norm, ws.best));
  const unsigned grid = (unsigned)std::min<int64_t>((int64_t)dm.L * ws.items_per_layer, 2048);
  OMNIMEM_LAUNCH(ws, K_GRAM, st, gram_max<T, D><<<grid, 256, 0, st>>>(desc, dm, on_keys, ws.pos, ws.counts,
                                       ws.inv_norm, ws.items, ws.n_items, ws.items_per_layer, ws.best));
  OMNIMEM_LAUNCH(ws, K_GRAM_FINISH, st, gram_finish<<<gtok, 256, 0, st>>>(desc, dm, ws.best, s));
}

}  // namespace

hipError_t launch_lists(const Dims& dm, const LayerDesc* desc, const Workspace& ws, int make_plan, hipStream_t st) {
  OMNIMEM_LAUNCH(ws, K_LISTS, st,
                 modality_lists<<<dm.L, 1024, 0, st>>>(desc, dm, ws.pos, ws.rank, ws.counts, ws.items, ws.n_items,
                                                       ws.items_per_layer, make_plan));
  return hipGetLastError();
}

hipError_t launch_redundancy(const Dims& dm, int dtype, int sim, int on_keys, const LayerDesc* desc,
                             const Workspace& ws, float* s, hipStream_t st) {
  hipError_t e = launch_lists(dm, desc, ws, sim == 0, st);
  if (e != hipSuccess) return e;
  if (dtype == 0) {
    if (dm.d == 128) launch_typed<uint16_t, 128>(dm, sim, on_keys, desc, ws, s, st);
    else launch_typed<uint16_t, 64>(dm, sim, on_keys, desc, ws, s, st);
  } else {
    if (dm.d == 128) launch_typed<float, 128>(dm, sim, on_keys, desc, ws, s, st);
    else launch_typed<float, 64>(dm, sim, on_keys, desc, ws, s, st);
  }
  return hipGetLastError();
}

}  // namespace omnimem
