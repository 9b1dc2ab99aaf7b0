// Cosine-similarity redundancy s_k (Eq. 7 of the OmniMem paper, computed
// from value vectors as Sec. 3.1 allows, or keys).
//
// Two modes:
//  SIM_MAX  s_k = max over the other rows j of k's (KV head, modality)
//           segment of cos(u_k, u_j).  lists_norms builds the segment's row
//           list (visual rows, then audio rows, each ascending) and fp32
//           inverse norms.  The Gram matrix U U^T is computed on MFMA in
//           256 x 64 tiles with fp32 accumulation and never leaves the chip:
//           for bf16 rows (gram_sym) each pair once, rows gathered through
//           the list by DMA, each product scaled into a cosine that enters
//           both rows' maxima; for fp32 rows (gram_pass) the whole matrix
//           over a copy of the rows in list order.  Maxima merge with
//           atomicMax on an order-preserving int encoding.
//  SIM_ADJ  Eq. (7) as printed: mean cosine with the previous and next row
//           of the same modality, in fp64.
#include "common.h"

namespace omnimem {

namespace {

// --- modality lists --------------------------------------------------------
// Per layer: pos[l][0][0 .. K_v) = visual rows ascending, pos[l][1][0 .. K_a)
// = audio rows ascending; rank[j] = index of row j inside its modality's
// list.  One workgroup per layer: a counting pass, one scan of the wave
// counts, and a placing pass.


__global__ __launch_bounds__(1024) void modality_lists(const LayerDesc* __restrict__ layers, Dims dm,
                                                      int* __restrict__ pos, int* __restrict__ rank,
                                                      int* __restrict__ counts) {
  const int l = blockIdx.x;
  const int N = layers[l].n;
  const uint8_t* mod = layers[l].mod;
  __shared__ int wave_tot[16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwaves = blockDim.x >> 6;
  const unsigned long long lt = (1ull << lane) - 1ull;
  int* Pv = pos + (int64_t)(2 * l) * list_stride(dm.max_tokens);
  int* Pa = Pv + list_stride(dm.max_tokens);
  int* R = rank + (int64_t)l * dm.max_tokens;
  // Wave w owns rows [w * 64S, (w + 1) * 64S); step i covers the 64
  // consecutive rows w * 64S + 64 i + lane, so reads and writes coalesce.
  const int S = (N + (int)blockDim.x - 1) / (int)blockDim.x;
  const int wrow0 = wave * 64 * S;
  constexpr int kGrp = 8;
  auto visual_group = [&](int i0, bool (&vis)[kGrp]) {
    int m[kGrp];  // branch-free reads (index clamped), all issued before the first use
#pragma unroll
    for (int u = 0; u < kGrp; ++u) m[u] = gload<uint8_t>(mod + min(wrow0 + (i0 + u) * 64 + lane, N - 1));
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      pin(m[u]);
      vis[u] = i0 + u < S && wrow0 + (i0 + u) * 64 + lane < N && m[u] == 0;
    }
  };
  int wv = 0;  // visual rows of this wave
  for (int i0 = 0; i0 < S; i0 += kGrp) {
    bool vis[kGrp];
    visual_group(i0, vis);
#pragma unroll
    for (int u = 0; u < kGrp; ++u) wv += __popcll(__ballot(vis[u]));
  }
  if (lane == 0) wave_tot[wave] = wv;
  __syncthreads();
  int vbase = 0, kv = 0;
  for (int w = 0; w < nwaves; ++w) {
    vbase += w < wave ? wave_tot[w] : 0;
    kv += wave_tot[w];
  }
  for (int i0 = 0, run = vbase; i0 < S; i0 += kGrp) {
    bool vis[kGrp];
    visual_group(i0, vis);
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      const int j = wrow0 + (i0 + u) * 64 + lane;
      const unsigned long long bal = __ballot(vis[u]);
      const int rv = run + __popcll(bal & lt);  // visual rows before j
      if (vis[u]) { Pv[rv] = j; R[j] = rv; }
      else if (i0 + u < S && j < N) { Pa[j - rv] = j; R[j] = j - rv; }
      run += __popcll(bal);
    }
  }
  if (threadIdx.x == 0) { counts[2 * l] = kv; counts[2 * l + 1] = N - kv; }
}

// 16 MFMAs: the 32-row block `row` of an LDS stage against two 32-column
// blocks of register operands; each LDS fragment feeds two MFMAs.
template <typename M, typename Tl, int NKS, typename T>
__device__ inline void mma_block(floatx16 (&acc)[2], const T* lds, int row, int half,
                                 const typename M::frag (&b)[2][NKS]) {
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    const typename M::frag f = Tl::template frag<M>(lds, row, ks, half);
    acc[0] = M::mma(f, b[0][ks], ks ? acc[0] : floatx16{});
    acc[1] = M::mma(f, b[1][ks], ks ? acc[1] : floatx16{});
  }
}

template <typename T, int D>
struct GatherShape {
  static constexpr int LPR = D * (int)sizeof(T) / 16;  // lanes per row
  static constexpr int RPB = 256 / LPR;                 // rows per workgroup
};

// --- modality lists, gathered rows and inverse norms in one pass ---------------
// For each (layer, KV head): perm[k] = u[row_k] with row_k the k-th row of
// the segment order [visual rows ascending | audio rows ascending], its
// inverse norm 1 / ||u|| in fp64 (0 for a zero row), and best[k] reset;
// with the lists that modality_lists makes.  Indexed by working-set row:
// each workgroup takes kListRows consecutive rows from j0 of one (layer, KV
// head), counts the visual rows of the whole layer and those
// before j0 from the modality mask itself, places its rows by a ballot
// prefix, and copies them to their segment positions with their inverse
// norms.  The workgroups of KV head 0 also write the lists (pos, rank,
// counts) for the later kernels.
constexpr int kListRows = 128;

template <typename T, int D, bool PERM>
__global__ __launch_bounds__(256) void lists_norms(const LayerDesc* __restrict__ layers, Dims dm, int on_keys,
                                                   int* __restrict__ pos, int* __restrict__ rank,
                                                   int* __restrict__ counts, T* __restrict__ perm,
                                                   float* __restrict__ inv, int* __restrict__ best) {
  const int l = blockIdx.z, g = blockIdx.y;
  const LayerDesc Ld = layers[l];
  const int N = Ld.n;
  const int j0 = blockIdx.x * kListRows;
  if (j0 >= N) return;  // the whole workgroup leaves together
  const uint8_t* mod = Ld.mod;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __shared__ int wv_before[4], wv_total[4];
  __shared__ int dst[kListRows];
  static_assert(kListRows % 64 == 0 && kListRows % 4 == 0, "whole waves of rows, word-aligned starts");
  // The rows' pieces and the rows' own mask bytes do not depend on the
  // counts: all are requested first, so that their latency overlaps the scan.
  constexpr int LPR = GatherShape<T, D>::LPR;
  constexpr int RPP = 256 / LPR;   // rows per pass
  constexpr int EPL = D / LPR;     // elements per lane
  static_assert(EPL * sizeof(T) == 16, "one 16-byte piece per lane");
  const int sub = threadIdx.x % LPR;
  const T* u = reinterpret_cast<const T*>(on_keys ? Ld.k : Ld.v) + (int64_t)g * Ld.kv_hs;
  constexpr int NP = kListRows / RPP;
  constexpr int NQ = kListRows / 64;
  uint4 v[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int r = p * RPP + (int)threadIdx.x / LPR;
    if (j0 + r < N) v[p] = gload16(u + (int64_t)(j0 + r) * Ld.kv_rs + sub * EPL);
  }
  int own[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int j = j0 + q * 64 + lane;
    own[q] = wave == 0 && j < N ? (int)gload<uint8_t>(mod + j) : 1;
  }
  // Visual rows before j0 and in the whole layer.  A 4-byte aligned mask is
  // read a word at a time (zero bytes counted with the haszero trick, j0
  // being a multiple of 4), eight words per thread in flight; the bytes of
  // a last partial word, or of an unaligned mask, one at a time.
  int before = 0, total = 0;
  const bool aligned = (reinterpret_cast<uintptr_t>(mod) & 3u) == 0;
  const int nw = aligned ? N / 4 : 0;
  const uint32_t* mw = reinterpret_cast<const uint32_t*>(mod);
  for (int w0 = (int)threadIdx.x * 8; w0 < nw; w0 += 256 * 8) {
    uint32_t w[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) w[u] = w0 + u < nw ? gload<uint32_t>(mw + w0 + u) : 0x01010101u;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint32_t z = ~(((w[u] & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | w[u] | 0x7F7F7F7Fu);  // 0x80 per zero byte
      const int c = __popc(z);
      total += c;
      before += 4 * (w0 + u) < j0 ? c : 0;
    }
  }
  for (int x = 4 * nw + (int)threadIdx.x; x < N; x += 256) {
    const int vis = gload<uint8_t>(mod + x) == 0;
    total += vis;
    before += x < j0 ? vis : 0;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    before += __shfl_xor(before, o, 64);
    total += __shfl_xor(total, o, 64);
  }
  if (lane == 0) { wv_before[wave] = before; wv_total[wave] = total; }
  __syncthreads();
  const int kv = wv_total[0] + wv_total[1] + wv_total[2] + wv_total[3];
  if (wave == 0) {  // the 64-row steps of the workgroup's rows, in order
    int vb = wv_before[0] + wv_before[1] + wv_before[2] + wv_before[3];
    int last[2] = {-1, -1};  // the last row of each list, if this workgroup holds it
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int j = j0 + q * 64 + lane;
      const bool in = j < N;
      const bool vis = in && own[q] == 0;
      const unsigned long long bal = __ballot(vis);
      const int rv = vb + __popcll(bal & ((1ull << lane) - 1ull));  // visual rows before j
      const int r = vis ? rv : j - rv;                              // rank inside the modality
      if (in) {
        dst[q * 64 + lane] = vis ? r : kv + r;
        if (g == 0) {
          pos[(int64_t)(2 * l + (vis ? 0 : 1)) * list_stride(dm.max_tokens) + r] = j;
          rank[(int64_t)l * dm.max_tokens + j] = r;
        }
        if (r == (vis ? kv : N - kv) - 1) last[vis ? 0 : 1] = j;
      }
      vb += __popcll(bal);
    }
    if (g == 0 && blockIdx.x == 0 && lane == 0) { counts[2 * l] = kv; counts[2 * l + 1] = N - kv; }
    if (g == 0) {  // each list's padding repeats its last row
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        const unsigned long long has = __ballot(last[m] >= 0);
        if (has) {
          const int jl = __shfl(last[m], __ffsll((long long)has) - 1, 64);
          int* pad = pos + (int64_t)(2 * l + m) * list_stride(dm.max_tokens) + (m ? N - kv : kv);
          for (int e = lane; e < kListPad; e += 64) pad[e] = jl;
        }
      }
    }
  }
  __syncthreads();
  // Pass p's row sum ends up in every lane of the row's group; lane sub = p
  // keeps it, so one fp64 square root and division per lane serves all NP
  // rows of the group (each is a long instruction sequence, paid per wave).
  static_assert(NP <= LPR, "a lane of the group for every pass");
  double mine = 0.0;
  int64_t omine = 0;
  bool in_mine = false;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int r = p * RPP + (int)threadIdx.x / LPR;
    const bool in = j0 + r < N;
    double acc = 0.0;
    int64_t o = 0;
    if (in) {
      o = ((int64_t)l * dm.Hkv + g) * dm.max_tokens + dst[r];
      if (PERM) *reinterpret_cast<uint4*>(perm + o * D + sub * EPL) = v[p];
      const uint32_t w[4] = {v[p].x, v[p].y, v[p].z, v[p].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if constexpr (sizeof(T) == 2) {
          const double a = __uint_as_float(w[e] << 16), b = __uint_as_float(w[e] & 0xFFFF0000u);
          acc += a * a + b * b;
        } else {
          const double a = __uint_as_float(w[e]);
          acc += a * a;
        }
      }
    }
#pragma unroll
    for (int x = LPR / 2; x > 0; x >>= 1) acc += __shfl_xor(acc, x, 64);
    if (sub == p) {
      mine = acc;
      omine = o;
      in_mine = in;
    }
  }
  if (in_mine) {
    inv[omine] = mine > 0.0 ? (float)(1.0 / sqrt(mine)) : 0.0f;
    best[omine] = kNoPartner;  // the Gram pass merges maxima into this
  }
}

// --- Gram max ------------------------------------------------------------------
// Work layout: a "row" is one block of 256 segment rows (4 waves x 64) held
// as MFMA B operands in registers; its "tiles" are all 64-row tiles of the
// same segment, streamed through LDS by DMA as A operands.  Rows of all
// segments (layer, KV head, modality) form one tile sequence, cut into
// chunks that the persistent workgroups take round-robin (as the score
// passes do).  The full matrix is computed, not its upper triangle: each
// row's maximum is then complete within its own register block, per lane
// (a lane holds one register row and 16 tile rows per 32-row block), with
// no cross-lane reduction or atomics per tile, no per-row norms in
// registers and one atomicMax per row per chunk.  Per element the work is
// dot * inv_j and a running maximum; inv_i scales the row's maximum once.
// Tile rows past the segment carry NaN inverse norms, which fmaxf ignores;
// a row's pair with itself is masked the same way.
constexpr int kGramBlock = 256;

// Tiles of a segment of K rows: every 256-row block sees all ceil(K/64).
__device__ inline int64_t gram_seg_tiles(int K) {
  const int64_t kt = (K + kScoreTile - 1) / kScoreTile, nb = (K + kGramBlock - 1) / kGramBlock;
  return nb * kt;
}

template <typename T, int D, bool BY_XCD>
__global__ __launch_bounds__(256, 2) void gram_pass(const LayerDesc* __restrict__ layers, Dims dm,
                                                    const int* __restrict__ counts, const T* __restrict__ perm,
                                                    const float* __restrict__ inv, int* __restrict__ best) {
  using M = Mfma<T>;
  using Tl = SwzTile<T, D>;
  constexpr int NKS = D / M::KSTEP;
  constexpr int kMaxL = 1024;
  __shared__ __attribute__((aligned(16))) T jt0[Tl::ELEMS];
  __shared__ __attribute__((aligned(16))) T jt1[Tl::ELEMS];
  __shared__ __attribute__((aligned(16))) float jinv[2][kScoreTile];
  __shared__ int64_t lbase[kMaxL + 1];  // first tile of each layer
  __shared__ int64_t sc[3];             // chunk size, total tiles, longest row

  // Tile bases of the layers and the chunking (as the score passes choose it).
  if (threadIdx.x == 0) {
    int64_t w = 0;
    int tmax = 0;
    for (int l = 0; l < dm.L; ++l) {
      lbase[l] = w;
      const int kv = counts[2 * l], ka = counts[2 * l + 1];
      w += (int64_t)dm.Hkv * (gram_seg_tiles(kv) + gram_seg_tiles(ka));
      tmax = max(tmax, (max(kv, ka) + kScoreTile - 1) / kScoreTile);
    }
    lbase[dm.L] = w;
    const int64_t P = gridDim.x, c_pref = max((int64_t)2 * tmax, (int64_t)32);
    int64_t c = 1;
    if (w > 0) {
      if (w <= P * c_pref) c = (w + P - 1) / P;
      else { const int64_t rounds = w / (P * c_pref); c = (w + P * rounds - 1) / (P * rounds); }
    }
    sc[0] = c;
    sc[1] = w;
    sc[2] = tmax;
  }
  __syncthreads();
  const int64_t c = sc[0], W = sc[1];
  const int i = gridDim.x % kXcds == 0 ? xcd_swizzle(blockIdx.x, gridDim.x) : (int)blockIdx.x;
  const int wave = wave_id(), lane = threadIdx.x & 63, half = lane >> 5;
  const typename Tl::Plan plan = Tl::plan(D);
  bool first = true;
  // Tiles [gt, gend) of the global sequence, row by row.
  auto run_range = [&](int64_t gt, const int64_t gend) {
    while (gt < gend) {
      // the row holding tile gt: layer, KV head, modality, register block
      int l = 0;
      for (int lo = 0, hi = dm.L - 1; lo < hi;) {
        const int mid = (lo + hi + 1) >> 1;
        if (lbase[mid] <= gt) lo = mid; else hi = mid - 1;
        l = lo;
      }
      const int kv = counts[2 * l], ka = counts[2 * l + 1];
      const int64_t tv = gram_seg_tiles(kv), tav = gram_seg_tiles(ka);
      int64_t rem = gt - lbase[l];
      const int g = (int)(rem / (tv + tav));
      rem -= g * (tv + tav);
      const int mu = rem >= tv ? 1 : 0;
      if (mu) rem -= tv;
      const int K = mu ? ka : kv;
      const int kt = (K + kScoreTile - 1) / kScoreTile;
      const int I = (int)(rem / kt);
      const int t0 = (int)(rem % kt);
      const int t1 = (int)min((int64_t)kt, t0 + (gend - gt));
      gt += t1 - t0;

      const int64_t seg_off = ((int64_t)l * dm.Hkv + g) * dm.max_tokens + (mu ? kv : 0);
      const T* U = perm + seg_off * D;
      const float* invs = inv + seg_off;
      if (!first) __syncthreads();  // every wave is done with the previous segment's stages
      first = false;

      auto tile_rows = [&](int t) { return min(kScoreTile, K - t * kScoreTile); };
      auto jinv_of = [&](int t) {  // inverse norm of tile row threadIdx.x (NaN past K)
        const int row = t * kScoreTile + (int)threadIdx.x;
        return row < K ? gload<float>(invs + row) : __builtin_nanf("");
      };
      // No load is waited for before the tile loop: the first tile's norms
      // and the register rows' own norms (for the final maxima) are held in
      // registers meanwhile.
      Tl::copy(jt0, U + (int64_t)t0 * kScoreTile * D, D, tile_rows(t0), plan);
      const float jinv_first = threadIdx.x < kScoreTile ? jinv_of(t0) : 0.0f;
      float jinv_next = 0.0f;
      if (t0 + 1 < t1) {
        Tl::copy(jt1, U + (int64_t)(t0 + 1) * kScoreTile * D, D, tile_rows(t0 + 1), plan);
        if (threadIdx.x < kScoreTile) jinv_next = jinv_of(t0 + 1);
      }
      // this wave's 64 register rows (two 32-column blocks of the output)
      const int c0 = I * kGramBlock + wave * 64;
      const float my_inv = gload<float>(invs + min(c0 + half * 32 + (lane & 31), K - 1));
      typename M::frag bf[2][NKS];
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) {
        const int my = min(c0 + cb * 32 + (lane & 31), K - 1);
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) bf[cb][ks] = M::gload(U + (int64_t)my * D + ks * M::KSTEP + half * M::PER_LANE);
      }
      float rmax[2] = {-INFINITY, -INFINITY};
      for (int t = t0; t < t1; ++t) {
        const int st = (t - t0) & 1;
        const T* cur = st ? jt1 : jt0;
        if (threadIdx.x < kScoreTile) jinv[st][threadIdx.x] = t > t0 ? jinv_next : jinv_first;
        dma_wait();
        __syncthreads();  // tile t and its norms landed; tile t-1's stage is free
        if (t > t0 && t + 1 < t1) {
          Tl::copy(st ? jt0 : jt1, U + (int64_t)(t + 1) * kScoreTile * D, D, tile_rows(t + 1), plan);
          if (threadIdx.x < kScoreTile) jinv_next = jinv_of(t + 1);
        }
        const bool diag = t * kScoreTile < c0 + 64 && c0 < (t + 1) * kScoreTile;
#pragma unroll
        for (int rb = 0; rb < 2; ++rb) {
          floatx16 acc[2];
          mma_block<M, Tl>(acc, cur, rb * 32 + (lane & 31), half, bf);
          float ij[16];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const floatx4 v = *reinterpret_cast<const floatx4*>(&jinv[st][rb * 32 + j * 8 + half * 4]);
            ij[j * 4 + 0] = v[0]; ij[j * 4 + 1] = v[1]; ij[j * 4 + 2] = v[2]; ij[j * 4 + 3] = v[3];
          }
          if (diag) {
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
              const int d = c0 + cb * 32 + (lane & 31) - (t * kScoreTile + rb * 32);
#pragma unroll
              for (int r = 0; r < 16; ++r) acc[cb][r] = acc_row(r, lane) == d ? __builtin_nanf("") : acc[cb][r];
            }
          }
#pragma unroll
          for (int cb = 0; cb < 2; ++cb) {
            float m = rmax[cb];
#pragma unroll
            for (int r = 0; r < 16; r += 2) m = fmaxf(m, fmaxf(acc[cb][r] * ij[r], acc[cb][r + 1] * ij[r + 1]));
            rmax[cb] = m;
          }
        }
      }
      // both lane halves hold different tile rows of the same register row
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) {
        const float m = fmaxf(rmax[cb], __shfl_xor(rmax[cb], 32, 64));
        const int row = c0 + cb * 32 + (lane & 31);
        if (half == cb && row < K && m > -INFINITY)
          atomicMax(best + seg_off + row, ord_f32(fminf(1.0f, fmaxf(-1.0f, m * my_inv))));
      }
    }
  };
  if constexpr (BY_XCD) {
    // Many (layer, KV head) units: unit u goes to the workgroups of XCD
    // u % 8.  They take the XCD's units k at a time (k units hold about one
    // longest row per workgroup) and split each group's tiles evenly, so an
    // XCD's L2 holds the rows of k units at a time instead of those of a
    // stretch of units spread over the whole chip.
    const int units = dm.L * dm.Hkv;
    const int px = (int)gridDim.x / kXcds, x = i / px, ix = i % px;
    const int64_t per0 = max((int64_t)1, W / max(units, 1));
    const int k = (int)max((int64_t)1, min((int64_t)8, (sc[2] * px + per0 - 1) / per0));
    for (int u0 = x; u0 < units; u0 += k * kXcds) {
      int64_t tot = 0;
      for (int jj = 0; jj < k && u0 + jj * kXcds < units; ++jj) {
        const int l = (u0 + jj * kXcds) / dm.Hkv;
        tot += gram_seg_tiles(counts[2 * l]) + gram_seg_tiles(counts[2 * l + 1]);
      }
      const int64_t cu = (tot + px - 1) / px, ga = ix * cu, gb = min(tot, ga + cu);
      int64_t off = 0;  // [ga, gb) of the concatenation of the group's tiles, unit by unit
      for (int jj = 0; jj < k && u0 + jj * kXcds < units && off < gb; ++jj) {
        const int u = u0 + jj * kXcds, l = u / dm.Hkv, g = u % dm.Hkv;
        const int64_t per = gram_seg_tiles(counts[2 * l]) + gram_seg_tiles(counts[2 * l + 1]);
        const int64_t lo = max(ga, off), hi = min(gb, off + per);
        if (lo < hi) run_range(lbase[l] + g * per + (lo - off), lbase[l] + g * per + (hi - off));
        off += per;
      }
    }
  } else {
    for (int64_t chunk = i; chunk * c < W; chunk += gridDim.x) run_range(chunk * c, min(W, chunk * c + c));
  }
}

// s in row order from the segment-order maxima.
__global__ void gram_finish(const LayerDesc* __restrict__ layers, Dims dm, const int* __restrict__ pos,
                            const int* __restrict__ counts, const int* __restrict__ best, float* __restrict__ s) {
  const int l = blockIdx.z, g = blockIdx.y;
  const int N = layers[l].n;
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= N) return;
  const int kv = counts[2 * l];
  const int64_t ls = list_stride(dm.max_tokens);
  const int row = k < kv ? pos[(int64_t)(2 * l) * ls + k] : pos[(int64_t)(2 * l + 1) * ls + k - kv];
  const int64_t o = ((int64_t)l * dm.Hkv + g) * dm.max_tokens;
  const int b = best[o + k];
  s[o + row] = b == kNoPartner ? 0.0f : fminf(1.0f, fmaxf(-1.0f, unord_f32(b)));
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
  const int* P = pos + (int64_t)(2 * l + mu) * list_stride(dm.max_tokens);
  const int t = rank[(int64_t)l * dm.max_tokens + j];
  const T* u = reinterpret_cast<const T*>(on_keys ? Ld.k : Ld.v) + (int64_t)g * Ld.kv_hs;
  const T* x = u + (int64_t)j * Ld.kv_rs;
  double sum = 0.0;
  int n = 0;
  if (t > 0) { sum += cos64<T, D>(x, u + (int64_t)P[t - 1] * Ld.kv_rs); ++n; }
  if (t + 1 < K) { sum += cos64<T, D>(x, u + (int64_t)P[t + 1] * Ld.kv_rs); ++n; }
  s[((int64_t)l * dm.Hkv + g) * dm.max_tokens + j] = n ? (float)(sum / n) : 0.0f;
}

// --- Eq. (7) as printed: on the layer's hidden states ------------------------
// One wave per working-set row j: the cosines of hidden state j with the
// previous and the next row of its modality (fp64 sums over the 16-byte
// pieces of the rows, lanes strided, then across the wave), their mean
// written to every KV head's row of s: hidden states are per token.
template <typename T>
__device__ inline void add_piece(const uint4& p, float (&out)[16 / sizeof(T)]) {
  const uint32_t w[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if constexpr (sizeof(T) == 2) {
      out[2 * e] = __uint_as_float(w[e] << 16);
      out[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    } else {
      out[e] = __uint_as_float(w[e]);
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void adjacent_cos_hidden(const LayerDesc* __restrict__ layers, Dims dm,
                                                           const int* __restrict__ pos, const int* __restrict__ rank,
                                                           const int* __restrict__ counts, float* __restrict__ s) {
  const int l = blockIdx.y;
  const LayerDesc Ld = layers[l];
  const int N = Ld.n;
  const int lane = threadIdx.x & 63;
  const int j = (int)blockIdx.x * 4 + wave_id();
  if (j >= N) return;  // the whole wave leaves
  const int mu = Ld.mod[j] ? 1 : 0;
  const int K = counts[2 * l + mu];
  const int* P = pos + (int64_t)(2 * l + mu) * list_stride(dm.max_tokens);
  const int t = rank[(int64_t)l * dm.max_tokens + j];
  const int jp = t > 0 ? P[t - 1] : -1, jn = t + 1 < K ? P[t + 1] : -1;
  const T* H = reinterpret_cast<const T*>(Ld.hidden);
  const T* x = H + (int64_t)j * Ld.hidden_rs;
  const T* xp = H + (int64_t)(jp < 0 ? j : jp) * Ld.hidden_rs;
  const T* xn = H + (int64_t)(jn < 0 ? j : jn) * Ld.hidden_rs;
  constexpr int EPP = 16 / (int)sizeof(T);  // elements per 16-byte piece
  const int pieces = dm.dh / EPP;
  double xx = 0.0, pp = 0.0, nn = 0.0, xpd = 0.0, xnd = 0.0;
  for (int c = lane; c < pieces; c += 64) {
    float a[EPP], b[EPP], d[EPP];
    add_piece<T>(gload16(x + c * EPP), a);
    add_piece<T>(gload16(xp + c * EPP), b);
    add_piece<T>(gload16(xn + c * EPP), d);
#pragma unroll
    for (int e = 0; e < EPP; ++e) {
      const double u = a[e], v = b[e], w = d[e];
      xx += u * u; pp += v * v; nn += w * w; xpd += u * v; xnd += u * w;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    xx += __shfl_xor(xx, o, 64);
    pp += __shfl_xor(pp, o, 64);
    nn += __shfl_xor(nn, o, 64);
    xpd += __shfl_xor(xpd, o, 64);
    xnd += __shfl_xor(xnd, o, 64);
  }
  auto cosv = [](double xy, double aa, double bb) {
    if (aa <= 0.0 || bb <= 0.0) return 0.0;
    const double c = xy / (sqrt(aa) * sqrt(bb));
    return c > 1.0 ? 1.0 : (c < -1.0 ? -1.0 : c);
  };
  double sum = 0.0;
  int n = 0;
  if (jp >= 0) { sum += cosv(xpd, xx, pp); ++n; }
  if (jn >= 0) { sum += cosv(xnd, xx, nn); ++n; }
  const float v = n ? (float)(sum / n) : 0.0f;
  for (int g = lane; g < dm.Hkv; g += 64) s[((int64_t)l * dm.Hkv + g) * dm.max_tokens + j] = v;
}

// --- all-pairs maximum on hidden states (Eq. 7's redundancy as the maximum
// cosine over all pairs of the modality, applied to them) ----
// d_model does not fit the register-resident operand of gram_pass, so both
// operands stream through LDS.  Work item: a pair (I <= J) of row blocks
// of one segment (layer, modality), rows gathered through the segment's row
// list; persistent workgroups take the pairs of all segments round-robin.
// The d axis goes by chunks of 64 (four MFMA k-steps), DMA-copied into two
// LDS stages (the next chunk lands while the current one is used).  The
// rows of the hidden states do not stay in L2, so the stages are fed at the
// bandwidth of the next cache level: the larger the block, the fewer bytes
// per MFMA.  Each wave owns 64 block rows and half the block's columns.  After the
// last chunk the products become cosines (inverse norms from LDS; a row's
// pair with itself and rows past the segment masked as NaN), and both the
// block rows' maxima (over the block's columns: halving exchanges across the
// lanes) and the columns' maxima (in-lane) are merged, first in LDS across
// waves, then into the rows' best values by atomicMax: each pair is
// computed once.
constexpr int kWideChunk = 64;  // d elements per LDS stage row
// Rows per block side: 256 for bf16 (eight waves, each a 64 x 128 tile; the
// double-buffered stage takes 128 KB, one workgroup per compute unit), 128
// for fp32 (four waves of 64 x 64; a 256-row fp32 stage would not fit LDS).
template <typename T> constexpr int wide_block() { return sizeof(T) == 2 ? 256 : 128; }
template <typename T> constexpr int wide_threads() { return wide_block<T>() / 32 * 64; }
// Waves per SIMD the register budget is sized for: two for bf16 (eight
// waves in the one workgroup of a compute unit); one for fp32 (four waves,
// and the stage leaves room for one workgroup).
template <typename T> constexpr int wide_waves_per_simd() { return sizeof(T) == 2 ? 2 : 1; }

__device__ inline float swz_xor(float v, int m) {
  // ds_swizzle bit mode (and-mask 0x1F, xor-mask m): within groups of 32 lanes
  switch (m) {
    case 16: return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x1F | (16 << 10)));
    case 8: return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x1F | (8 << 10)));
    case 4: return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x1F | (4 << 10)));
    case 2: return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x1F | (2 << 10)));
    default: return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x1F | (1 << 10)));
  }
}
// Maximum of w[r] over the 32 lanes of each half-wave, for every r: after
// halving exchanges (xor 16, 8, 4, 2, then 1) w[0] of lane k holds the
// maximum for r = (k >> 1) & 15, in lanes k and k ^ 1 alike.
__device__ inline void half_wave_max16(float (&w)[16], int lane) {
#pragma unroll
  for (int m = 16, n = 16; m >= 2; m >>= 1, n >>= 1) {
    const bool hi = (lane & m) != 0;
#pragma unroll
    for (int i = 0; i < n / 2; ++i) {
      const float send = hi ? w[i] : w[i + n / 2];
      const float keep = hi ? w[i + n / 2] : w[i];
      w[i] = fmaxf(keep, swz_xor(send, m));
    }
  }
  w[0] = fmaxf(w[0], swz_xor(w[0], 1));
}

// inv[l][j] = 1 / ||h_j|| (fp64 sum of squares; 0 for a zero row) and best
// reset, one wave per working-set row.
template <typename T>
__global__ __launch_bounds__(256) void hidden_norms(const LayerDesc* __restrict__ layers, Dims dm,
                                                    float* __restrict__ inv, int* __restrict__ best) {
  const int l = blockIdx.y;
  const LayerDesc Ld = layers[l];
  const int j = (int)blockIdx.x * 4 + wave_id(), lane = threadIdx.x & 63;
  if (j >= Ld.n) return;
  constexpr int EPP = 16 / (int)sizeof(T);
  const T* x = reinterpret_cast<const T*>(Ld.hidden) + (int64_t)j * Ld.hidden_rs;
  double ss = 0.0;
  for (int c = lane; c < dm.dh / EPP; c += 64) {
    float a[EPP];
    add_piece<T>(gload16(x + c * EPP), a);
#pragma unroll
    for (int e = 0; e < EPP; ++e) ss += (double)a[e] * a[e];
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  if (lane == 0) {
    inv[(int64_t)l * dm.max_tokens + j] = ss > 0.0 ? (float)(1.0 / sqrt(ss)) : 0.0f;
    best[(int64_t)l * dm.max_tokens + j] = kNoPartner;
  }
}

template <typename T>
__global__ __launch_bounds__(wide_threads<T>(), wide_waves_per_simd<T>()) void gram_wide(
    const LayerDesc* __restrict__ layers, Dims dm, const int* __restrict__ pos, const int* __restrict__ counts,
    const float* __restrict__ inv, int* __restrict__ best) {
  using M = Mfma<T>;
  using Tl = SwzTile<T, kWideChunk>;  // one stage tile: 64 rows of a 64-element chunk
  constexpr int BR = wide_block<T>();
  constexpr int kThr = wide_threads<T>();
  constexpr int TPS = BR / kScoreTile;  // stage tiles per block side
  constexpr int WC = BR / 2;            // block columns per wave
  constexpr int CB = WC / 32;           // 32-column MFMA blocks per wave
  constexpr int KS = kWideChunk / M::KSTEP;
  constexpr int EPC = 16 / (int)sizeof(T);
  constexpr int CPR = kWideChunk / EPC;  // 16-byte pieces per stage row
  constexpr int kMaxSegs = 2048;
  __shared__ __attribute__((aligned(16))) T stage[2][2 * TPS][Tl::ELEMS];  // [buffer][A tiles, B tiles]
  __shared__ int seg_first[kMaxSegs + 1];  // first pair of each segment (pair counts fit 31 bits)
  __shared__ float inv_a[BR], inv_b[BR];
  __shared__ int row_a[BR], row_b[BR];
  __shared__ int mx_a[BR], mx_b[BR];
  const int S = 2 * dm.L;
  for (int q = threadIdx.x; q < S; q += blockDim.x) {
    const int nb = (counts[q] + BR - 1) / BR;
    seg_first[q + 1] = nb * (nb + 1) / 2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    seg_first[0] = 0;
    for (int q = 0; q < S; ++q) seg_first[q + 1] += seg_first[q];
  }
  __syncthreads();
  const int total = uniform(seg_first[S]);
  const int w = wave_id(), lane = threadIdx.x & 63, half = lane >> 5;
  const int wr = w >> 1, wc = w & 1;  // the wave's 64 block rows (A) and WC block columns (B)
  const int nchunks = dm.dh / kWideChunk;
  // Rounds of gridDim.x pairs; in each, XCD x (blockIdx % 8) takes a run of
  // consecutive pairs, which mostly share their first block, so its L2
  // serves that block's chunks to all of them.  A last partial round is
  // split evenly over the XCDs.  (A grid that is not a multiple of 8 takes
  // pairs in plain order.)
  const bool by_xcd = gridDim.x % kXcds == 0;
  for (int base = 0; base < total; base += gridDim.x) {
    const int R = min((int)gridDim.x, total - base);
    const int per = by_xcd ? (R + kXcds - 1) / kXcds : R;
    const int k = by_xcd ? (int)blockIdx.x / kXcds : (int)blockIdx.x;
    const int p = base + (by_xcd ? ((int)blockIdx.x % kXcds) * per : 0) + k;
    if (k >= per || p >= base + R) continue;  // uniform over the workgroup
    // segment and block pair of p
    int q = 0;
    for (int lo = 0, hi = S - 1; lo < hi;) {
      const int mid = (lo + hi + 1) >> 1;
      if (uniform(seg_first[mid]) <= p) lo = mid; else hi = mid - 1;
      q = lo;
    }
    const int l = q >> 1;
    const int K = counts[q];
    const int nb = (K + BR - 1) / BR;
    int r = p - uniform(seg_first[q]);
    int bi = 0;
    while (r >= nb - bi) { r -= nb - bi; ++bi; }
    const int bj = bi + r;
    const LayerDesc Ld = layers[l];
    const int* P = pos + (int64_t)q * list_stride(dm.max_tokens);
    __syncthreads();  // every wave is done with the previous pair's LDS
    for (int t = threadIdx.x; t < 2 * BR; t += blockDim.x) {
      const int side = t / BR, k = t % BR;
      const int m = (side ? bj : bi) * BR + k;
      const int row = P[min(m, K - 1)];
      const float iv = m < K ? inv[(int64_t)l * dm.max_tokens + row] : __builtin_nanf("");
      if (side) { row_b[k] = row; inv_b[k] = iv; mx_b[k] = kNoPartner; }
      else { row_a[k] = row; inv_a[k] = iv; mx_a[k] = kNoPartner; }
    }
    __syncthreads();
    // this thread's DMA pieces of a chunk: 2 TPS tiles x 64 rows x CPR pieces
    // over the workgroup
    constexpr int kInstrPerTile = kScoreTile * CPR / 64;
    constexpr int kPieces = 2 * TPS * kInstrPerTile / (kThr / 64);
    const T* H = reinterpret_cast<const T*>(Ld.hidden);
    const T* src[kPieces];
#pragma unroll
    for (int u = 0; u < kPieces; ++u) {
      const int J = w * kPieces + u;  // DMA instruction of the workgroup
      const int tile = J / kInstrPerTile, slot = (J % kInstrPerTile) * 64 + lane;
      const int rr = slot / CPR, c = (slot % CPR) ^ (rr & (CPR - 1));
      const int k = (tile % TPS) * kScoreTile + rr;
      const int row = tile < TPS ? row_a[k] : row_b[k];
      src[u] = H + (int64_t)row * Ld.hidden_rs + c * EPC;
    }
    // Copies of chunk ch into stage buffer buf, issued with dma16_opaque: the
    // compiler does not see them write LDS, so reads of the other buffer do
    // not wait for them (a buffer is read only after dma_wait and a barrier).
    auto dma_chunk = [&](int ch, int buf) {
#pragma unroll
      for (int u = 0; u < kPieces; ++u) {
        const int J = w * kPieces + u;
        const int tile = J / kInstrPerTile, jt = J % kInstrPerTile;
        dma16_opaque(src[u] + ch * kWideChunk, &stage[buf][tile][jt * 64 * EPC]);
      }
    };
    floatx16 acc[2][CB];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) acc[rb][cb] = floatx16{};
    dma_chunk(0, 0);
    for (int ch = 0; ch < nchunks; ++ch) {
      const int buf = ch & 1;
      dma_wait();
      __syncthreads();  // chunk ch landed; every wave is done with the other stage
      if (ch + 1 < nchunks) dma_chunk(ch + 1, buf ^ 1);
      const T* A = stage[buf][wr];  // the wave's 64 A rows: tile wr
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        typename M::frag fa[2], fb[CB];
#pragma unroll
        for (int x = 0; x < 2; ++x) fa[x] = Tl::template frag<M>(A, x * 32 + (lane & 31), ks, half);
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {  // B column block wc * WC + cb * 32
          const int bc = wc * WC + cb * 32;
          fb[cb] = Tl::template frag<M>(stage[buf][TPS + bc / kScoreTile], bc % kScoreTile + (lane & 31), ks, half);
        }
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int cb = 0; cb < CB; ++cb) acc[rb][cb] = M::mma(fa[rb], fb[cb], acc[rb][cb]);
      }
    }
    // cosines; row (A) maxima across the lanes, column (B) maxima in-lane
    float cmax[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) cmax[cb] = -INFINITY;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      float wv[16];
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) wv[rr] = -INFINITY;
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        const int jb = wc * WC + cb * 32 + (lane & 31);  // block column
        const float ib = inv_b[jb];
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int ia_k = wr * 64 + rb * 32 + acc_row(rr, lane);  // block row
          float c = acc[rb][cb][rr] * inv_a[ia_k] * ib;
          if (bi == bj && ia_k == jb) c = __builtin_nanf("");
          wv[rr] = fmaxf(wv[rr], c);
          cmax[cb] = fmaxf(cmax[cb], c);
        }
      }
      half_wave_max16(wv, lane);
      const int rr = (lane >> 1) & 15;
      const int ia_k = wr * 64 + rb * 32 + acc_row(rr, lane);
      if ((lane & 1) == 0 && wv[0] > -INFINITY) atomicMax(&mx_a[ia_k], ord_f32(fminf(1.0f, fmaxf(-1.0f, wv[0]))));
    }
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
      const float m = fmaxf(cmax[cb], __shfl_xor(cmax[cb], 32, 64));
      const int jb = wc * WC + cb * 32 + (lane & 31);
      if (half == 0 && m > -INFINITY) atomicMax(&mx_b[jb], ord_f32(fminf(1.0f, fmaxf(-1.0f, m))));
    }
    __syncthreads();
    for (int t = threadIdx.x; t < 2 * BR; t += blockDim.x) {
      const int side = t / BR, k = t % BR;
      const int m = (side ? bj : bi) * BR + k;
      const int v = side ? mx_b[k] : mx_a[k];
      if (m < K && v != kNoPartner) atomicMax(best + (int64_t)l * dm.max_tokens + (side ? row_b[k] : row_a[k]), v);
    }
  }
}

// s[l][g][j] of every KV head from the hidden states' maxima.
__global__ void hidden_finish(const LayerDesc* __restrict__ layers, Dims dm, const int* __restrict__ best,
                              float* __restrict__ s) {
  const int l = blockIdx.y;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= layers[l].n) return;
  const int b = best[(int64_t)l * dm.max_tokens + j];
  const float v = b == kNoPartner ? 0.0f : fminf(1.0f, fmaxf(-1.0f, unord_f32(b)));
  for (int g = 0; g < dm.Hkv; ++g) s[((int64_t)l * dm.Hkv + g) * dm.max_tokens + j] = v;
}

// --- Gram max, each pair once (bf16 keys or values) -----------------------------
// Work layout: a "row" is one block I of 256 segment rows (4 waves x 64)
// held in registers as MFMA A operands; its tiles are the 64-row tiles
// t >= 4I of the same segment (the block's own rows and every later row),
// copied by DMA through the segment's row list straight from the key or
// value rows into LDS, where they are B operands.  So each pair of rows
// (i, j) with block(i) <= block(j) is computed once: by the register block of
// i against the tile of j.  A product becomes a cosine, (dot * inv_j) * inv_i,
// which enters two maxima: the register row's (a running maximum per lane
// over the tile rows the lane holds, reduced across lanes once per row of
// work) and the tile row's (over the lane's 32 register rows in-lane, then
// over lane halves and waves through LDS, merged into best once per tile).
// Inside a wave, the MFMAs of one 32-row column block of a tile run while
// the previous column block's products become cosines, across the per-tile
// barrier (the score passes' software pipeline).  Register rows and tile
// rows past the segment carry NaN inverse norms, and a row's pair with itself
// is set to NaN; fmaxf ignores both.
constexpr int kSymBlock = 256;

// Tiles of a segment of K rows: register block I sees tiles 4I .. kt-1.
__device__ inline int64_t sym_seg_tiles(int K) {
  const int64_t kt = (K + kScoreTile - 1) / kScoreTile, nb = (K + kSymBlock - 1) / kSymBlock;
  return nb * kt - 2 * nb * (nb - 1);
}

__device__ inline void gatomic_max(int* p, int v) {
  typedef __attribute__((address_space(1))) int global_int;
  __hip_atomic_fetch_max((global_int*)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// v_max_f32 / v_max3_f32 written out: a running maximum carried across loop
// iterations is not known to be canonical, so fmaxf would first quiet it with
// an extra v_max_f32 per use.  In IEEE mode these return the other operand
// for a quiet NaN input, the only NaN that reaches them here.
__device__ inline float vmax(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ inline float vmax3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// One phase of gram_sym in a wave: with MMA, the MFMAs (k-steps x the two
// register row blocks) of the 32 tile rows from LDS row `brow` into `out`;
// with EPI, interleaved with them (32 / (2 NKS) per MFMA), the products of
// the previous column block `in` become cosines and enter the row maxima
// `rmax` and the column maximum `cm`.  LDS fragments are requested two
// k-steps ahead of their MFMAs.
template <int NKS, bool MMA, bool EPI>
__device__ inline void sym_phase(floatx16 (&out)[2], bf16x8 (&a)[2][NKS], const uint16_t* lds, int brow, int half,
                                 floatx16 (&in)[2], float invj, float (&iv)[2][16], float (&rmax)[2][16],
                                 float& cm) {
  using M = Mfma<uint16_t>;
  using Tl = SwzTile<uint16_t, NKS * 16>;
  constexpr int NG = 2 * NKS;     // groups, one MFMA each
  constexpr int PER = 32 / NG;    // cosines per group
  static_assert(PER * NG == 32 && PER >= 1, "products per lane of a column block");
  // LDS address of row brow's k-step-ks fragment in the swizzled tile: piece
  // (2 ks + half) ^ (brow & XM) of the row, that is base ^ (ks << 5) with
  // base the k-step-0 address (the tile starts on a ROWB boundary and the
  // row's own offset has no bits below ROWB).  The base is rebuilt per
  // phase rather than held across the tile loop.
  static_assert(Tl::ROWB >= 32 * NKS, "k-step bits stay inside a row");
  typedef __attribute__((address_space(3))) const bf16x8 lds_frag;
  uint32_t base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)lds + brow * Tl::ROWB +
                  ((half ^ (brow & Tl::XM)) << 4);
  pin(base);
  auto frag = [&](int ks) { return *(lds_frag*)(uintptr_t)(base ^ (uint32_t)(ks << 5)); };
  bf16x8 f[NKS];
  if (MMA) __builtin_amdgcn_s_setprio(1);  // a wave in its MFMA stream issues ahead of one in the tile bookkeeping
  if (MMA) {
    f[0] = frag(0);
    if (NKS > 1) f[1] = frag(1);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int ks = g >> 1, rb = g & 1;
    if (MMA) {
      if (rb == 0 && ks + 2 < NKS) f[ks + 2] = frag(ks + 2);
      pin(a[rb][ks]);
      out[rb] = M::mma(a[rb][ks], f[ks], ks ? out[rb] : floatx16{});
    }
    if (EPI) {
      float c[PER];
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int e = g * PER + i, erb = e >> 4, r = e & 15;
        c[i] = in[erb][r] * invj * iv[erb][r];
        rmax[erb][r] = vmax(rmax[erb][r], c[i]);
        pin(rmax[erb][r]);
      }
#pragma unroll
      for (int i = 0; i < PER; i += 2) cm = vmax3(cm, c[i], c[i + 1]);
      pin(cm);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  if (MMA) __builtin_amdgcn_s_setprio(0);
}

template <int D, bool BY_XCD>
__global__ __launch_bounds__(256, 2) void gram_sym(const LayerDesc* __restrict__ layers, Dims dm, int on_keys,
                                                   const int* __restrict__ counts, const int* __restrict__ pos,
                                                   const float* __restrict__ inv, int* __restrict__ best) {
  using T = uint16_t;
  using M = Mfma<T>;
  using Tl = SwzTile<T, D>;
  constexpr int NKS = D / M::KSTEP;
  constexpr int IPW = Tl::INSTR_PER_WAVE;  // DMA copies per wave and tile
  constexpr int kMaxL = 1024;
  constexpr int kSlots = 4;  // column maxima of tiles t - 1 (being merged) .. t + 2 (being written)
  __shared__ __attribute__((aligned(256))) T jt[2][Tl::ELEMS];  // stages start on row boundaries
  __shared__ float cmx[kSlots][4][2][kScoreTile];  // [tile][wave][lane half][tile row]
  __shared__ int64_t lbase[kMaxL + 1];  // first tile of each layer
  __shared__ int64_t sc[2];             // total tiles, longest row

  if (threadIdx.x == 0) {
    int64_t w = 0;
    int tmax = 0;
    for (int l = 0; l < dm.L; ++l) {
      lbase[l] = w;
      const int kv = counts[2 * l], ka = counts[2 * l + 1];
      w += (int64_t)dm.Hkv * (sym_seg_tiles(kv) + sym_seg_tiles(ka));
      tmax = max(tmax, (max(kv, ka) + kScoreTile - 1) / kScoreTile);
    }
    lbase[dm.L] = w;
    sc[0] = w;
    sc[1] = tmax;
  }
  __syncthreads();
  const int64_t W = sc[0];
  const int i = gridDim.x % kXcds == 0 ? xcd_swizzle(blockIdx.x, gridDim.x) : (int)blockIdx.x;
  const int wave = wave_id(), lane = threadIdx.x & 63, half = lane >> 5;
  // This lane's DMA pieces of a tile: copy j moves piece ln % CPR of tile
  // row (wave * IPW + j) * RPI + ln / CPR (RPI rows per copy) to its
  // swizzled place, piece (ln % CPR) ^ (row & XM); the rows come through the
  // row list.  As wave * IPW * RPI is a multiple of XM + 1, the swizzle is
  // the lane's own, ((ln % CPR) ^ (ln / CPR)) << 4 bytes, xor the copy's
  // ((j * RPI) & XM) << 4.  (Recomputed where used: cheaper than registers
  // held across the tile loop.)
  constexpr int RPI = 64 / Tl::CPR;
  static_assert((IPW * RPI) % (Tl::XM + 1) == 0 && RPI <= Tl::XM + 1, "copy swizzle is per lane");
  bool first = true;

  auto run_range = [&](int64_t gt, const int64_t gend) {
    while (gt < gend) {
      // the row holding tile gt: layer, KV head, modality, register block
      int l = 0;
      for (int lo = 0, hi = dm.L - 1; lo < hi;) {
        const int mid = (lo + hi + 1) >> 1;
        if (lbase[mid] <= gt) lo = mid; else hi = mid - 1;
        l = lo;
      }
      const int kv = counts[2 * l], ka = counts[2 * l + 1];
      const int64_t tv = sym_seg_tiles(kv), tav = sym_seg_tiles(ka);
      int64_t rem = gt - lbase[l];
      const int g = (int)(rem / (tv + tav));
      rem -= g * (tv + tav);
      const int mu = rem >= tv ? 1 : 0;
      if (mu) rem -= tv;
      const int K = mu ? ka : kv;
      const int kt = (K + kScoreTile - 1) / kScoreTile;
      int I = 0;
      while (rem >= kt - 4 * I) { rem -= kt - 4 * I; ++I; }
      const int t0 = 4 * I + (int)rem;
      const int t1 = (int)min((int64_t)kt, t0 + (gend - gt));
      gt += t1 - t0;

      const LayerDesc& Ld = layers[l];
      const T* U = reinterpret_cast<const T*>(on_keys ? Ld.k : Ld.v) + (int64_t)g * Ld.kv_hs;
      const int64_t rs = Ld.kv_rs;
      const int* P = pos + (int64_t)(2 * l + mu) * list_stride(dm.max_tokens);
      const int64_t seg_off = ((int64_t)l * dm.Hkv + g) * dm.max_tokens + (mu ? kv : 0);
      const float* invs = inv + seg_off;
      int* bst = best + seg_off;
      if (!first) __syncthreads();  // every wave is done with the previous row's stages and maxima
      first = false;

      int pr[IPW];  // source rows of this lane's pieces of the next tile to copy
      // (byte offsets of rows in one head fit 31 bits, which the entry points check)
      const uint32_t rs_b = (uint32_t)(rs * (int64_t)sizeof(T));
      // (rows past the segment come from the list's padding, which repeats its last row)
      auto rows_of = [&](int t) {
        int ln = lane;
        pin(ln);
        const int* Pt = P + (t * kScoreTile + wave * IPW * RPI);
#pragma unroll
        for (int j = 0; j < IPW; ++j) pr[j] = gload<int>(Pt + ((uint32_t)ln / Tl::CPR + j * RPI));
      };
      auto copy = [&](int buf) {
        int ln = lane;
        pin(ln);
        const uint32_t colb = (((uint32_t)ln % Tl::CPR) ^ ((uint32_t)ln / Tl::CPR)) << 4;
#pragma unroll
        for (int j = 0; j < IPW; ++j)
          dma16_opaque_s(U, __umul24((uint32_t)pr[j], rs_b) + (colb ^ (uint32_t)(((j * RPI) & Tl::XM) << 4)),
                         &jt[buf][(wave * IPW + j) * 64 * Tl::EPC]);
      };
      auto invj_of = [&](int t, int cb) {  // inverse norm of tile row t*64 + cb*32 + lane%32 (NaN past K)
        const int row = t * kScoreTile + cb * 32 + (lane & 31);
        const float v = gload<float>(invs + (uint32_t)min(row, K - 1));
        return row < K ? v : __builtin_nanf("");
      };
      rows_of(t0);
      copy(0);
      if (t0 + 1 < t1) { rows_of(t0 + 1); copy(1); }
      if (t0 + 2 < t1) rows_of(t0 + 2);
      // this wave's 64 register rows (two 32-row blocks of the output)
      const int c0 = I * kSymBlock + wave * 64;
      bf16x8 a[2][NKS];
      float iv[2][16], rmax[2][16];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        const int src = gload<int>(P + (uint32_t)(c0 + rb * 32 + (lane & 31)));
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
          a[rb][ks] = M::gload(U + ((uint32_t)src * (uint32_t)rs + ks * M::KSTEP + half * M::PER_LANE));
        int ln = lane;
        pin(ln);  // the rows below are recomputed per row of work, not held across the loop
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = c0 + rb * 32 + acc_row(r, ln);
          const float v = gload<float>(invs + (uint32_t)min(row, K - 1));
          iv[rb][r] = row < K ? v : __builtin_nanf("");
          rmax[rb][r] = -INFINITY;
        }
      }
      float ij[2] = {invj_of(t0, 0), invj_of(t0, 1)}, ijn[2] = {0.0f, 0.0f};
      // a column block of tile t that holds the register rows of block rb: the pairs (i, i) are dropped
      // (lane's column m = lane % 32 is row acc_row(r) for r = 4 (q / 8) + q % 4, q = m - 4 half, if q >= 0
      // and q % 8 < 4; the register index is computed where it is used, not held across the loop)
      auto mask_diag = [&](floatx16 (&acc)[2], int t, int cb) {
        const int col0 = t * kScoreTile + cb * 32;
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
          if (col0 == c0 + rb * 32) {
            int q = (lane & 31) - half * 4;
            pin(q);
            const int rd = q >= 0 && (q & 4) == 0 ? ((q >> 3) << 2) | (q & 3) : -1;
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[rb][r] = r == rd ? __builtin_nanf("") : acc[rb][r];
          }
      };
      auto merge = [&](int t) {  // tile t's row maxima over the register block into best, by wave t % 4
        if (wave == (t & 3)) {
          float m = -INFINITY;
#pragma unroll
          for (int w = 0; w < 4; ++w) m = fmaxf(m, fmaxf(cmx[t & 3][w][0][lane], cmx[t & 3][w][1][lane]));
          const int row = t * kScoreTile + lane;
          if (row < K && m > -INFINITY) gatomic_max(bst + row, ord_f32(fminf(1.0f, fmaxf(-1.0f, m))));
        }
      };
      floatx16 acc0[2], acc1[2];
      float cm = -INFINITY;
      dma_wait();
      __syncthreads();  // tiles t0 and t0+1 landed
      sym_phase<NKS, true, false>(acc0, a, jt[0], lane & 31, half, acc1, 0.0f, iv, rmax, cm);
      // phase A of tile t: MFMAs of its tile rows 32..63 || cosines of its rows 0..31
      auto phase_a = [&](int t) {
        mask_diag(acc0, t, 0);
        cm = -INFINITY;
        sym_phase<NKS, true, true>(acc1, a, jt[(t - t0) & 1], 32 + (lane & 31), half, acc0, ij[0], iv, rmax, cm);
        cmx[t & 3][wave][half][lane & 31] = cm;
      };
      for (int t = t0; t + 1 < t1; ++t) {
        const int st = (t - t0) & 1;
        ijn[0] = invj_of(t + 1, 0);
        ijn[1] = invj_of(t + 1, 1);
        phase_a(t);
        dma_wait();
        __syncthreads();  // tile t+1 landed; every wave is done with tile t's stage
        pin(ijn[0]);
        pin(ijn[1]);
        if (t + 2 < t1) {
          copy(st);
          if (t + 3 < t1) rows_of(t + 3);
        }
        if (t > t0) merge(t - 1);
        // phase B: MFMAs of tile rows 0..31 of tile t+1 || cosines of rows 32..63 of tile t
        mask_diag(acc1, t, 1);
        cm = -INFINITY;
        sym_phase<NKS, true, true>(acc0, a, jt[st ^ 1], lane & 31, half, acc1, ij[1], iv, rmax, cm);
        cmx[t & 3][wave][half][32 + (lane & 31)] = cm;
        ij[0] = ijn[0];
        ij[1] = ijn[1];
      }
      {  // the last tile: its phase B has no MFMAs
        const int t = t1 - 1;
        phase_a(t);
        __syncthreads();
        if (t > t0) merge(t - 1);
        mask_diag(acc1, t, 1);
        cm = -INFINITY;
        sym_phase<NKS, false, true>(acc0, a, jt[0], 0, half, acc1, ij[1], iv, rmax, cm);
        cmx[t & 3][wave][half][32 + (lane & 31)] = cm;
      }
      __syncthreads();  // the last tile's maxima are in LDS
      merge(t1 - 1);
      // the register rows' maxima: over the 32 lanes of each half
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        half_wave_max16(rmax[rb], lane);
        const int row = c0 + rb * 32 + acc_row((lane >> 1) & 15, lane);
        if ((lane & 1) == 0 && row < K && rmax[rb][0] > -INFINITY)
          gatomic_max(bst + row, ord_f32(fminf(1.0f, fmaxf(-1.0f, rmax[rb][0]))));
      }
    }
  };
  // Unit u = (layer, KV head) goes to XCD u % 8 (with BY_XCD; otherwise the
  // whole grid is one group), whose workgroups take its units k at a time
  // and split their tiles evenly, so that an XCD's L2 holds the rows of k
  // units at a time.  One call site of run_range keeps one copy of its code.
  constexpr int kX = BY_XCD ? kXcds : 1;
  const int units = dm.L * dm.Hkv;
  const int px = (int)gridDim.x / kX, x = i / px, ix = i % px;
  const int64_t per0 = max((int64_t)1, W / max(units, 1));
  const int k = (int)max((int64_t)1, min((int64_t)8, (sc[1] * px + per0 - 1) / per0));
  for (int u0 = x; u0 < units; u0 += k * kX) {
    int64_t tot = 0;
    for (int jj = 0; jj < k && u0 + jj * kX < units; ++jj) {
      const int l = (u0 + jj * kX) / dm.Hkv;
      tot += sym_seg_tiles(counts[2 * l]) + sym_seg_tiles(counts[2 * l + 1]);
    }
    const int64_t cu = (tot + px - 1) / px, ga = ix * cu, gb = min(tot, ga + cu);
    int64_t off = 0;
    for (int jj = 0; jj < k && u0 + jj * kX < units && off < gb; ++jj) {
      const int u = u0 + jj * kX, l = u / dm.Hkv, g = u % dm.Hkv;
      const int64_t per = sym_seg_tiles(counts[2 * l]) + sym_seg_tiles(counts[2 * l + 1]);
      const int64_t lo = max(ga, off), hi = min(gb, off + per);
      if (lo < hi) run_range(lbase[l] + g * per + (lo - off), lbase[l] + g * per + (hi - off));
      off += per;
    }
  }
}

template <typename T, int D>
void launch_typed(const Dims& dm, int sim, int on_keys, const LayerDesc* desc, const Workspace& ws, float* s,
                  hipStream_t st) {
  const dim3 gtok((unsigned)((dm.max_tokens + 255) / 256), dm.Hkv, dm.L);
  if (sim == 1) {
    OMNIMEM_LAUNCH(ws, K_ADJ, st, adjacent_cos<T, D><<<gtok, 256, 0, st>>>(desc, dm, on_keys, ws.pos, ws.rank, ws.counts, s));
    return;
  }
  const dim3 glist((unsigned)((dm.max_tokens + kListRows - 1) / kListRows), dm.Hkv, dm.L);
  T* perm = reinterpret_cast<T*>(ws.perm);
  const bool by_xcd = dm.L * dm.Hkv >= 2 * kXcds && ws.gram_grid % kXcds == 0;
  if constexpr (sizeof(T) == 2) {  // bf16: each pair once, rows gathered through the row lists
    OMNIMEM_LAUNCH(ws, K_NORMS, st,
                   lists_norms<T, D, false><<<glist, 256, 0, st>>>(desc, dm, on_keys, ws.pos, ws.rank, ws.counts,
                                                                   perm, ws.inv_norm, ws.best));
    if (by_xcd)
      OMNIMEM_LAUNCH(ws, K_GRAM_SYM, st,
                     gram_sym<D, true><<<ws.gram_grid, 256, 0, st>>>(desc, dm, on_keys, ws.counts, ws.pos,
                                                                      ws.inv_norm, ws.best));
    else
      OMNIMEM_LAUNCH(ws, K_GRAM_SYM, st,
                     gram_sym<D, false><<<ws.gram_grid, 256, 0, st>>>(desc, dm, on_keys, ws.counts, ws.pos,
                                                                       ws.inv_norm, ws.best));
    OMNIMEM_LAUNCH(ws, K_GRAM_FINISH, st, gram_finish<<<gtok, 256, 0, st>>>(desc, dm, ws.pos, ws.counts, ws.best, s));
    return;
  }
  OMNIMEM_LAUNCH(ws, K_NORMS, st,
                 lists_norms<T, D, true><<<glist, 256, 0, st>>>(desc, dm, on_keys, ws.pos, ws.rank, ws.counts, perm,
                                                                ws.inv_norm, ws.best));
  if (by_xcd)
    OMNIMEM_LAUNCH(ws, K_GRAM, st,
                   gram_pass<T, D, true><<<ws.gram_grid, 256, 0, st>>>(desc, dm, ws.counts, perm, ws.inv_norm, ws.best));
  else
    OMNIMEM_LAUNCH(ws, K_GRAM, st,
                   gram_pass<T, D, false><<<ws.gram_grid, 256, 0, st>>>(desc, dm, ws.counts, perm, ws.inv_norm, ws.best));
  OMNIMEM_LAUNCH(ws, K_GRAM_FINISH, st, gram_finish<<<gtok, 256, 0, st>>>(desc, dm, ws.pos, ws.counts, ws.best, s));
}

}  // namespace

hipError_t launch_lists(const Dims& dm, const LayerDesc* desc, const Workspace& ws, hipStream_t st) {
  OMNIMEM_LAUNCH(ws, K_LISTS, st, modality_lists<<<dm.L, 1024, 0, st>>>(desc, dm, ws.pos, ws.rank, ws.counts));
  return hipGetLastError();
}

hipError_t launch_redundancy(const Dims& dm, int dtype, int sim, int source, const LayerDesc* desc,
                             const Workspace& ws, float* s, hipStream_t st) {
  if (sim == 1) {  // the all-pairs mode computes the lists inside lists_norms
    hipError_t e = launch_lists(dm, desc, ws, st);
    if (e != hipSuccess) return e;
  }
  if (source == 2 && sim == 0) {  // hidden states, all pairs
    hipError_t e = launch_lists(dm, desc, ws, st);
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)((dm.max_tokens + 3) / 4), dm.L);
    const dim3 gtok((unsigned)((dm.max_tokens + 255) / 256), dm.L);
    if (dtype == 0) {
      OMNIMEM_LAUNCH(ws, K_NORMS_H, st, hidden_norms<uint16_t><<<grid, 256, 0, st>>>(desc, dm, ws.inv_norm, ws.best));
      OMNIMEM_LAUNCH(ws, K_GRAM_H, st,
                     gram_wide<uint16_t><<<ws.gram_grid / 2, wide_threads<uint16_t>(), 0, st>>>(
                         desc, dm, ws.pos, ws.counts, ws.inv_norm, ws.best));
    } else {
      OMNIMEM_LAUNCH(ws, K_NORMS_H, st, hidden_norms<float><<<grid, 256, 0, st>>>(desc, dm, ws.inv_norm, ws.best));
      OMNIMEM_LAUNCH(ws, K_GRAM_H, st,
                     gram_wide<float><<<ws.gram_grid, wide_threads<float>(), 0, st>>>(desc, dm, ws.pos, ws.counts,
                                                                                      ws.inv_norm, ws.best));
    }
    OMNIMEM_LAUNCH(ws, K_FINISH_H, st, hidden_finish<<<gtok, 256, 0, st>>>(desc, dm, ws.best, s));
    return hipGetLastError();
  }
  if (source == 2) {  // hidden states, adjacent
    const dim3 grid((unsigned)((dm.max_tokens + 3) / 4), dm.L);
    if (dtype == 0)
      OMNIMEM_LAUNCH(ws, K_ADJ_H, st, adjacent_cos_hidden<uint16_t><<<grid, 256, 0, st>>>(desc, dm, ws.pos, ws.rank,
                                                                                       ws.counts, s));
    else
      OMNIMEM_LAUNCH(ws, K_ADJ_H, st, adjacent_cos_hidden<float><<<grid, 256, 0, st>>>(desc, dm, ws.pos, ws.rank,
                                                                                    ws.counts, s));
    return hipGetLastError();
  }
  const int on_keys = source == 1 ? 1 : 0;
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
