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
// Per layer: pos[0 .. K_v) = visual rows ascending, pos[K_v .. N) = audio
// rows ascending; rank[j] = index of row j inside its modality's list.
__global__ __launch_bounds__(1024) void modality_lists(const LayerDesc* __restrict__ layers, Dims dm,
                                                      int* __restrict__ pos, int* __restrict__ rank,
                                                      int* __restrict__ counts) {
  const int l = blockIdx.x;
  const LayerDesc Ld = layers[l];
  const int N = Ld.n;
  const uint8_t* mod = Ld.mod;
  __shared__ int wave_tot[16];
  __shared__ int s_total;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwaves = blockDim.x >> 6;

  // total visual rows
  int cnt = 0;
  for (int j = threadIdx.x; j < N; j += blockDim.x) cnt += (mod[j] == 0);
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
  if (lane == 0) wave_tot[wave] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int t = 0;
    for (int w = 0; w < nwaves; ++w) t += wave_tot[w];
    s_total = t;
  }
  __syncthreads();
  const int kv = s_total;
  int* P = pos + (int64_t)l * dm.max_tokens;
  int* R = rank + (int64_t)l * dm.max_tokens;
  int base = 0;  // visual rows before the current tile
  for (int t0 = 0; t0 < N; t0 += blockDim.x) {
    const int j = t0 + threadIdx.x;
    const bool vis = j < N && mod[j] == 0;
    const unsigned long long bal = __ballot(vis);
    const int before = __popcll(bal & ((1ull << lane) - 1ull));
    __syncthreads();
    if (lane == 0) wave_tot[wave] = __popcll(bal);
    __syncthreads();
    int wbase = base;
    for (int w = 0; w < wave; ++w) wbase += wave_tot[w];
    if (j < N) {
      const int rv = wbase + before;   // visual rows before j
      if (vis) { P[rv] = j; R[j] = rv; }
      else { const int ra = j - rv; P[kv + ra] = j; R[j] = ra; }
    }
    int tile = 0;
    for (int w = 0; w < nwaves; ++w) tile += wave_tot[w];
    base += tile;
  }
  if (threadIdx.x == 0) { counts[2 * l] = kv; counts[2 * l + 1] = N - kv; }
}

// --- Gram work plan ----------------------------------------------------------
// Segment (l, g, mu) with T = ceil(K / 128) row blocks owns, for each row
// block I, ceil((T - I) / S) items covering column blocks [J0, J0 + S).
// F(n) = sum_{m=1..n} ceil(m / S) counts the items of rows with n blocks.
__device__ inline int64_t plan_F(int64_t n) {
  const int64_t q = n / kGramStrip, r = n % kGramStrip;
  return kGramStrip * q * (q + 1) / 2 + r * (q + 1);
}

__global__ __launch_bounds__(256) void gram_plan(Dims dm, const int* __restrict__ counts,
                                                 int4* __restrict__ items, int* __restrict__ n_items,
                                                 int64_t cap) {
  const int nseg = dm.L * dm.Hkv * 2;
  __shared__ int64_t s_base;
  if (threadIdx.x == 0) s_base = 0;
  __syncthreads();
  for (int seg = 0; seg < nseg; ++seg) {
    const int l = seg / (dm.Hkv * 2), mu = seg & 1;
    const int K = counts[2 * l + mu];
    const int T = (K + kGramTile - 1) / kGramTile;
    const int64_t base = s_base;
    const int64_t FT = plan_F(T);
    for (int I = threadIdx.x; I < T; I += blockDim.x) {
      int64_t off = base + FT - plan_F(T - I);
      for (int J0 = I; J0 < T; J0 += kGramStrip, ++off)
        if (off < cap) items[off] = make_int4(seg, I, J0, min(T, J0 + kGramStrip));
    }
    __syncthreads();
    if (threadIdx.x == 0) s_base = base + FT;
    __syncthreads();
  }
  if (threadIdx.x == 0) *n_items = (int)min(s_base, cap);
}

// --- inverse norms -----------------------------------------------------------
// inv_norm[l][g][j] = 1 / ||u_j|| (0 for a zero row), accumulated in fp64.
template <typename T, int D>
__global__ __launch_bounds__(256) void inv_norms(const LayerDesc* __restrict__ layers, Dims dm, int on_keys,
                                                 float* __restrict__ inv) {
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
  if (row < N && sub == 0) inv[((int64_t)l * dm.Hkv + g) * dm.max_tokens + row] = acc > 0.0 ? (float)(1.0 / sqrt(acc)) : 0.0f;
}

__global__ void fill_int(int* __restrict__ p, int64_t n, int v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = v;
}

// --- Gram max -------------------------------------------------------------
// One work item = row block I of a segment against column blocks [J0, J1).
// Wave w computes the 64 x 64 quadrant (w >> 1, w & 1) of each 128 x 128
// tile as 2 x 2 MFMA tiles.  Column maxima are reduced per tile and merged
// at once; row maxima are carried across the strip and merged at the end.
template <typename T, int D>
__global__ __launch_bounds__(256) void gram_max(const LayerDesc* __restrict__ layers, Dims dm, int on_keys,
                                                const int* __restrict__ pos, const int* __restrict__ counts,
                                                const float* __restrict__ inv, const int4* __restrict__ items,
                                                const int* __restrict__ n_items, int* __restrict__ best) {
  using M = Mfma<T>;
  constexpr int NKS = D / M::KSTEP;
  constexpr int LD = D + lds_pad<T>();
  constexpr int TB = kGramTile;
  __shared__ __attribute__((aligned(16))) T tI[TB * LD];
  __shared__ __attribute__((aligned(16))) T tJ[TB * LD];
  __shared__ float invI[TB], invJ[TB];
  __shared__ int rowsI[TB], rowsJ[TB];

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, half = lane >> 5;
  const int wr = wave >> 1, wc = wave & 1;
  const int total = *n_items;

  for (int it = blockIdx.x; it < total; it += gridDim.x) {
    const int4 item = items[it];
    const int seg = item.x, I = item.y, J0 = item.z, J1 = item.w;
    const int l = seg / (dm.Hkv * 2), g = (seg >> 1) % dm.Hkv, mu = seg & 1;
    const LayerDesc Ld = layers[l];
    const int K = counts[2 * l + mu];
    const int* P = pos + (int64_t)l * dm.max_tokens + (mu ? counts[2 * l] : 0);
    const T* u = reinterpret_cast<const T*>(on_keys ? Ld.k : Ld.v) + (int64_t)g * Ld.kv_hs;
    const float* inv_g = inv + ((int64_t)l * dm.Hkv + g) * dm.max_tokens;
    int* best_g = best + ((int64_t)l * dm.Hkv + g) * dm.max_tokens;

    __syncthreads();  // previous item done with the LDS tiles
    const int validI = min(TB, K - I * TB);
    if (threadIdx.x < TB) {
      const int r = threadIdx.x;
      const int row = r < validI ? P[I * TB + r] : 0;
      rowsI[r] = row;
      invI[r] = r < validI ? inv_g[row] : 0.0f;
    }
    __syncthreads();
    stage_rows_gather<T, D>(tI, u, Ld.kv_rs, rowsI, TB, validI);

    float rmax[2][16];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int r = 0; r < 16; ++r) rmax[rt][r] = -INFINITY;

    for (int J = J0; J < J1; ++J) {
      const int validJ = min(TB, K - J * TB);
      __syncthreads();
      if (threadIdx.x < TB) {
        const int r = threadIdx.x;
        const int row = r < validJ ? P[J * TB + r] : 0;
        rowsJ[r] = row;
        invJ[r] = r < validJ ? inv_g[row] : 0.0f;
      }
      __syncthreads();
      stage_rows_gather<T, D>(tJ, u, Ld.kv_rs, rowsJ, TB, validJ);
      __syncthreads();

      floatx16 acc[2][2];
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int ct = 0; ct < 2; ++ct) acc[rt][ct] = floatx16{};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        typename M::frag af[2], bf[2];
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
          af[rt] = M::load(tI + (wr * 64 + rt * 32 + (lane & 31)) * LD + ks * M::KSTEP + half * M::PER_LANE);
#pragma unroll
        for (int ct = 0; ct < 2; ++ct)
          bf[ct] = M::load(tJ + (wc * 64 + ct * 32 + (lane & 31)) * LD + ks * M::KSTEP + half * M::PER_LANE);
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int ct = 0; ct < 2; ++ct) acc[rt][ct] = M::mma(af[rt], bf[ct], acc[rt][ct]);
      }

      // Exclude the diagonal and the padding rows/columns of ragged blocks.
      const bool masked = (I == J) || validI < TB || validJ < TB;
      float ri[2][16];
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int r = 0; r < 16; ++r) ri[rt][r] = invI[wr * 64 + rt * 32 + acc_row(r, lane)];
      float cmax[2];
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) {
        const int cj = wc * 64 + ct * 32 + (lane & 31);
        const float ij = invJ[cj];
        float cm = -INFINITY;
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int ri_ = wr * 64 + rt * 32 + acc_row(r, lane);
            float dot = acc[rt][ct][r];
            if (masked && (ri_ >= validI || cj >= validJ || (I == J && ri_ == cj))) dot = -INFINITY;
            cm = fmaxf(cm, dot * ri[rt][r]);
            rmax[rt][r] = fmaxf(rmax[rt][r], dot * ij);
          }
        cmax[ct] = cm;
      }
      // Column maxima: combine the two row halves, scale, merge globally.
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) {
        float cm = fmaxf(cmax[ct], __shfl_xor(cmax[ct], 32, 64));
        const int cj = wc * 64 + ct * 32 + (lane & 31);
        if (half == ct && cj < validJ && cm != -INFINITY) {
          const float c = fminf(1.0f, fmaxf(-1.0f, cm * invJ[cj]));
          atomicMax(best_g + rowsJ[cj], ord_f32(c));
        }
      }
    }
    // Row maxima: reduce across the 32 lanes that share each row.
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v = rmax[rt][r];
#pragma unroll
        for (int o = 16; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
        rmax[rt][r] = v;
      }
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ri_ = wr * 64 + rt * 32 + acc_row(r, lane);
        // lane (lane & 31) == r writes row r of its half
        if ((lane & 31) == r && ri_ < validI && rmax[rt][r] != -INFINITY) {
          const float c = fminf(1.0f, fmaxf(-1.0f, rmax[rt][r] * invI[ri_]));
          atomicMax(best_g + rowsI[ri_], ord_f32(c));
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
  const int* P = pos + (int64_t)l * dm.max_tokens + (mu ? counts[2 * l] : 0);
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
  OMNIMEM_LAUNCH(ws, K_PLAN, st, gram_plan<<<1, 256, 0, st>>>(dm, ws.counts, ws.items, ws.n_items, ws.items_cap));
  const dim3 gnorm((unsigned)((dm.max_tokens + 15) / 16), dm.Hkv, dm.L);
  OMNIMEM_LAUNCH(ws, K_NORMS, st, inv_norms<T, D><<<gnorm, 256, 0, st>>>(desc, dm, on_keys, ws.inv_norm));
  const int64_t nbest = (int64_t)dm.L * dm.Hkv * dm.max_tokens;
  OMNIMEM_LAUNCH(ws, K_FILL, st, fill_int<<<(unsigned)std::min<int64_t>((nbest + 255) / 256, 4096), 256, 0, st>>>(ws.best, nbest, kNoPartner));
  const unsigned grid = (unsigned)std::min<int64_t>(ws.items_cap, 2048);
  OMNIMEM_LAUNCH(ws, K_GRAM, st, gram_max<T, D><<<grid, 256, 0, st>>>(desc, dm, on_keys, ws.pos, ws.counts,
                                       ws.inv_norm, ws.items, ws.n_items, ws.best));
  OMNIMEM_LAUNCH(ws, K_GRAM_FINISH, st, gram_finish<<<gtok, 256, 0, st>>>(desc, dm, ws.best, s));
}

}  // namespace

hipError_t launch_lists(const Dims& dm, const LayerDesc* desc, const Workspace& ws, hipStream_t st) {
  OMNIMEM_LAUNCH(ws, K_LISTS, st, modality_lists<<<dm.L, 1024, 0, st>>>(desc, dm, ws.pos, ws.rank, ws.counts));
  return hipGetLastError();
}

hipError_t launch_redundancy(const Dims& dm, int dtype, int sim, int on_keys, const LayerDesc* desc,
                             const Workspace& ws, float* s, hipStream_t st) {
  hipError_t e = launch_lists(dm, desc, ws, st);
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
