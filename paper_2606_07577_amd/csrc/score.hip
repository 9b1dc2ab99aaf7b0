// Accumulated attention importance a_k (Eq. 6 of the OmniMem paper).
//
// a[g][j] sums, over every chunk query i of every query head h of KV head
// g, the softmax probability A[h][i][j] of the chunk attention (Eq. 1:
// one softmax over both caches and the visible chunk rows).  A row of A is
// only known once its normaliser is, so the work is two passes over the
// score matrix S = scale * Q K^T, both on MFMA tiles:
//   lse_pass     per (head, query): log sum_j exp(S[i][j]), online max/sum
//   colsum_pass  per (head, key):   sum_i exp(S[i][j] - lse[i])
//   head_sum     a[g][j] = sum over the G query heads of KV head g.
// Scores stay in registers; nothing of size queries x keys touches HBM.
#include "common.h"

namespace omnimem {

namespace {

constexpr int kThreads = 256;     // 4 wavefronts
constexpr int kLseQ = 128;        // queries per lse workgroup (32 per wave)
constexpr int kLseK = 64;         // keys per LDS stage in lse_pass
constexpr int kColK = 256;        // keys per colsum workgroup (64 per wave)
constexpr int kColQ = 64;         // queries per LDS stage in colsum_pass

__device__ inline float wave_xor32(float x) {
  return __shfl_xor(x, 32, 64);
}

// Pass 1: lse[h][i] for the 128 queries [q0, q0+128) of head h in layer l.
// MFMA tile: rows = 32 keys (A from LDS), columns = 32 queries (B in
// registers), so each lane owns one query and 16 of its keys per tile.
template <typename T, int D>
__global__ __launch_bounds__(kThreads) void lse_pass(const LayerDesc* __restrict__ layers, Dims dm,
                                                     float* __restrict__ lse_buf) {
  using M = Mfma<T>;
  constexpr int NKS = D / M::KSTEP;
  constexpr int LD = D + lds_pad<T>();
  __shared__ __attribute__((aligned(16))) T ktile[kLseK * LD];

  const int l = blockIdx.z, h = blockIdx.y;
  const LayerDesc Ld = layers[l];
  const int C = Ld.n_chunk, N = Ld.n, nc = Ld.n_cache;
  const int q0 = blockIdx.x * kLseQ;
  if (q0 >= C) return;
  float* out = lse_buf + ((int64_t)l * dm.Hq + h) * dm.max_chunk;
  if (Ld.lse_in) {  // caller supplied the normalisers: copy them through
    for (int i = q0 + threadIdx.x; i < min(C, q0 + kLseQ); i += blockDim.x)
      out[i] = Ld.lse_in[(int64_t)h * C + i];
    return;
  }
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, half = lane >> 5;
  const int g = h / dm.G;
  const T* q = reinterpret_cast<const T*>(Ld.q) + (int64_t)h * Ld.q_hs;
  const T* k = reinterpret_cast<const T*>(Ld.k) + (int64_t)g * Ld.kv_hs;
  const int qw = q0 + wave * 32;           // first query of this wave
  const int my_q = qw + (lane & 31);

  typename M::frag qf[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks)
    qf[ks] = (my_q < C) ? M::load(q + (int64_t)my_q * Ld.q_rs + ks * M::KSTEP + half * M::PER_LANE)
                        : M::zero();

  // Keys any query of the block can see, and those of this wave.
  const int kend_blk = dm.causal ? min(N, nc + min(q0 + kLseQ, C)) : N;
  const int kend_wave = dm.causal ? min(N, nc + min(qw + 32, C)) : N;
  const float sl2 = Ld.scale_log2;
  float m = -1e30f, lsum = 0.0f;

  for (int kt = 0; kt < kend_blk; kt += kLseK) {
    __syncthreads();
    stage_rows<T, D>(ktile, k + (int64_t)kt * Ld.kv_rs, Ld.kv_rs, kLseK, min(kLseK, N - kt));
    __syncthreads();
    if (qw >= C) continue;
#pragma unroll
    for (int rb = 0; rb < kLseK / 32; ++rb) {
      const int kb = kt + rb * 32;
      if (kb >= kend_wave) break;
      floatx16 acc = {};
      const T* arow = ktile + (rb * 32 + (lane & 31)) * LD + half * M::PER_LANE;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) acc = M::mma(M::load(arow + ks * M::KSTEP), qf[ks], acc);
      // Masking is needed when the tile reaches past N or past some query's
      // causal horizon (key row nc + t is visible to query i iff t <= i).
      const bool edge = (kb + 32 > N) || (dm.causal && kb + 31 - nc > qw);
      float x[16];
      float mloc = -1e30f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        x[r] = acc[r] * sl2;
        if (edge) {
          const int key = kb + acc_row(r, lane);
          const bool vis = key < N && (!dm.causal || key < nc || key - nc <= my_q);
          x[r] = vis ? x[r] : -INFINITY;
        }
        mloc = fmaxf(mloc, x[r]);
      }
      const float mnew = fmaxf(m, mloc);
      float add = 0.0f;
#pragma unroll
      for (int r = 0; r < 16; ++r) add += __builtin_amdgcn_exp2f(x[r] - mnew);
      lsum = lsum * __builtin_amdgcn_exp2f(m - mnew) + add;
      m = mnew;
    }
  }
  // Lanes l and l ^ 32 hold the same query's two key halves.
  const float m2 = wave_xor32(m), l2 = wave_xor32(lsum);
  const float mt = fmaxf(m, m2);
  const float lt = lsum * __builtin_amdgcn_exp2f(m - mt) + l2 * __builtin_amdgcn_exp2f(m2 - mt);
  if (half == 0 && my_q < C) out[my_q] = (mt + __log2f(lt)) * kLn2;
}

// Pass 2: per-query-head column sums part[h][j] = sum_i exp(S[i][j] - lse[i])
// for the 256 keys [k0, k0+256).  MFMA tile: rows = 32 queries (A from LDS),
// columns = 32 keys (B in registers, two column blocks per wave), so each
// lane accumulates one key's sum over 16 query rows per tile.
template <typename T, int D>
__global__ __launch_bounds__(kThreads) void colsum_pass(const LayerDesc* __restrict__ layers, Dims dm,
                                                        const float* __restrict__ lse_buf,
                                                        float* __restrict__ part) {
  using M = Mfma<T>;
  constexpr int NKS = D / M::KSTEP;
  constexpr int LD = D + lds_pad<T>();
  __shared__ __attribute__((aligned(16))) T qtile[kColQ * LD];
  __shared__ __attribute__((aligned(16))) float lse2[kColQ];

  const int l = blockIdx.z, h = blockIdx.y;
  const LayerDesc Ld = layers[l];
  const int C = Ld.n_chunk, N = Ld.n, nc = Ld.n_cache;
  const int k0 = blockIdx.x * kColK;
  if (k0 >= N) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, half = lane >> 5;
  const int g = h / dm.G;
  const T* q = reinterpret_cast<const T*>(Ld.q) + (int64_t)h * Ld.q_hs;
  const T* k = reinterpret_cast<const T*>(Ld.k) + (int64_t)g * Ld.kv_hs;
  const float* lse = lse_buf + ((int64_t)l * dm.Hq + h) * dm.max_chunk;
  const int kw = k0 + wave * 64;  // first key of this wave

  typename M::frag kf[2][NKS];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    const int key = kw + cb * 32 + (lane & 31);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      kf[cb][ks] = key < N ? M::load(k + (int64_t)key * Ld.kv_rs + ks * M::KSTEP + half * M::PER_LANE)
                           : M::zero();
  }
  // First query that sees any key of the block: chunk row nc + t is seen
  // by queries i >= t.
  const int qstart = dm.causal ? max(0, k0 - nc) : 0;
  const int qfirst_wave = dm.causal ? max(0, kw - nc) : 0;
  const float sl2 = Ld.scale_log2;
  float cs0 = 0.0f, cs1 = 0.0f;

  for (int qt = (qstart / kColQ) * kColQ; qt < C; qt += kColQ) {
    __syncthreads();
    stage_rows<T, D>(qtile, q + (int64_t)qt * Ld.q_rs, Ld.q_rs, kColQ, min(kColQ, C - qt));
    if (threadIdx.x < kColQ) {
      const int i = qt + threadIdx.x;
      lse2[threadIdx.x] = i < C ? lse[i] * kLog2e : INFINITY;
    }
    __syncthreads();
    if (kw >= N) continue;
#pragma unroll
    for (int rb = 0; rb < kColQ / 32; ++rb) {
      const int qb = qt + rb * 32;
      if (qb >= C || qb + 31 < qfirst_wave) continue;
      floatx16 acc0 = {}, acc1 = {};
      const T* arow = qtile + (rb * 32 + (lane & 31)) * LD + half * M::PER_LANE;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const typename M::frag af = M::load(arow + ks * M::KSTEP);
        acc0 = M::mma(af, kf[0][ks], acc0);
        acc1 = M::mma(af, kf[1][ks], acc1);
      }
      // lse2 of the 16 query rows this lane holds: 4 runs of 4 rows.
      float lrow[16];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const floatx4 v = *reinterpret_cast<const floatx4*>(lse2 + rb * 32 + j * 8 + half * 4);
        lrow[j * 4 + 0] = v[0]; lrow[j * 4 + 1] = v[1]; lrow[j * 4 + 2] = v[2]; lrow[j * 4 + 3] = v[3];
      }
      const bool edge = dm.causal && (kw + 63 - nc > qb);
      if (!edge) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          cs0 += __builtin_amdgcn_exp2f(acc0[r] * sl2 - lrow[r]);
          cs1 += __builtin_amdgcn_exp2f(acc1[r] * sl2 - lrow[r]);
        }
      } else {
        const int t0 = kw + (lane & 31) - nc, t1 = t0 + 32;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = qb + acc_row(r, lane);
          const float p0 = __builtin_amdgcn_exp2f(acc0[r] * sl2 - lrow[r]);
          const float p1 = __builtin_amdgcn_exp2f(acc1[r] * sl2 - lrow[r]);
          cs0 += (t0 <= i) ? p0 : 0.0f;
          cs1 += (t1 <= i) ? p1 : 0.0f;
        }
      }
    }
  }
  cs0 += wave_xor32(cs0);
  cs1 += wave_xor32(cs1);
  float* out = part + ((int64_t)l * dm.Hq + h) * dm.max_tokens;
  const int key = kw + half * 32 + (lane & 31);
  if (key < N) out[key] = half ? cs1 : cs0;
}

// a[l][g][j] = sum over the G query heads of KV head g, in head order.
__global__ void head_sum(const LayerDesc* __restrict__ layers, Dims dm, const float* __restrict__ part,
                         float* __restrict__ a) {
  const int l = blockIdx.z, g = blockIdx.y;
  const int N = layers[l].n;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= N) return;
  const float* p = part + ((int64_t)l * dm.Hq + (int64_t)g * dm.G) * dm.max_tokens + j;
  float sum = 0.0f;
  for (int hh = 0; hh < dm.G; ++hh) sum += p[(int64_t)hh * dm.max_tokens];
  a[((int64_t)l * dm.Hkv + g) * dm.max_tokens + j] = sum;
}

template <typename T, int D>
void launch_typed(const Dims& dm, const LayerDesc* desc, const Workspace& ws, float* lse_buf, float* a,
                  hipStream_t st) {
  dim3 g1((unsigned)((dm.max_chunk + kLseQ - 1) / kLseQ), dm.Hq, dm.L);
  OMNIMEM_LAUNCH(ws, K_LSE, st, lse_pass<T, D><<<g1, kThreads, 0, st>>>(desc, dm, lse_buf));
  dim3 g2((unsigned)((dm.max_tokens + kColK - 1) / kColK), dm.Hq, dm.L);
  OMNIMEM_LAUNCH(ws, K_COLSUM, st, colsum_pass<T, D><<<g2, kThreads, 0, st>>>(desc, dm, lse_buf, ws.part));
  dim3 g3((unsigned)((dm.max_tokens + 255) / 256), dm.Hkv, dm.L);
  OMNIMEM_LAUNCH(ws, K_HEADSUM, st, head_sum<<<g3, 256, 0, st>>>(desc, dm, ws.part, a));
}

}  // namespace

hipError_t launch_score(const Dims& dm, int dtype, const LayerDesc* desc, const Workspace& ws,
                        float* lse_buf, float* a, int /*need_lse*/, hipStream_t st) {
  if (dtype == 0) {
    if (dm.d == 128) launch_typed<uint16_t, 128>(dm, desc, ws, lse_buf, a, st);
    else launch_typed<uint16_t, 64>(dm, desc, ws, lse_buf, a, st);
  } else {
    if (dm.d == 128) launch_typed<float, 128>(dm, desc, ws, lse_buf, a, st);
    else launch_typed<float, 64>(dm, desc, ws, lse_buf, a, st);
  }
  return hipGetLastError();
}

}  // namespace omnimem
