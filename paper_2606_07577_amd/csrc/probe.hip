// Throughput probes of the instruction mixes the score passes run (built as
// libomnimem_probe.so, used only for measurement).  Each kernel keeps every
// SIMD busy with independent work for `iters` iterations and writes one value
// per lane only when `flag` is set (it never is), so nothing is optimised
// away and nothing but registers (and, in one probe, LDS) is touched.
//
//   probe_mfma      four independent chains of v_mfma_f32_32x32x16_bf16
//   probe_exp       sixteen independent chains of v_exp_f32
//   probe_mix       the per-MFMA work of the LSE pass at head_dim 128: per
//                   phase, 16 MFMAs into one accumulator pair while the 32
//                   scores per lane of the other pair go through FMA (scale,
//                   reference), exp2 and a running sum (two of each per
//                   MFMA), software-pipelined as in the pass
//   probe_mix_lds   the same, with the MFMA's key fragments read from LDS
//                   (one ds_read_b128 per k-step and phase), as in the pass
//   probe_mix_bar   probe_mix_lds with one workgroup barrier every two
//                   phases (one per 64-key tile, as in the pass)
//   probe_gram      the per-MFMA work of the bf16 Gram pass at head_dim 128:
//                   per phase, 16 MFMAs (two register row blocks, k-step
//                   fragments of the tile rows read from LDS two k-steps
//                   ahead) while the 32 products per lane of the other
//                   accumulator pair become cosines (two multiplies) and
//                   enter a running row maximum and a column maximum
//                   (v_max3 over pairs); one barrier every two phases
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

template <typename V>
__device__ inline void pin(V& v) { asm volatile("" : "+v"(v)); }

__device__ inline floatx16 mma(bf16x8 a, bf16x8 b, floatx16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ inline bf16x8 frag_of(int seed) {
  bf16x8 f;
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] = (__bf16)(0.001f * (float)((seed + i) & 7));
  return f;
}

constexpr int NKS = 8;   // k-steps of one 32x32 tile at head_dim 128

__global__ __launch_bounds__(256) void probe_mfma(int iters, float* out, int flag) {
  const bf16x8 a = frag_of(threadIdx.x), b = frag_of(threadIdx.x + 3);
  floatx16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int it = 0; it < iters; ++it) {
    c0 = mma(a, b, c0);
    c1 = mma(a, b, c1);
    c2 = mma(a, b, c2);
    c3 = mma(a, b, c3);
  }
  if (flag) out[blockIdx.x * blockDim.x + threadIdx.x] = c0[0] + c1[1] + c2[2] + c3[3];
}

__global__ __launch_bounds__(256) void probe_exp(int iters, float* out, int flag) {
  float x[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) x[i] = 0.01f * (float)(threadIdx.x + i);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 16; ++i) x[i] = __builtin_amdgcn_exp2f(-x[i]);  // stays in (0, 1]
  }
  float t = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) t += x[i];
  if (flag) out[blockIdx.x * blockDim.x + threadIdx.x] = t;
}

// One phase: MFMAs into `o` (two query columns x NKS k-steps) interleaved
// with the exp/sum work on `in`, as the LSE pass schedules it.
template <bool LDS>
__device__ inline void mix_phase(floatx16 (&o)[2], const floatx16 (&in)[2], bf16x8 (&f)[NKS],
                                 bf16x8 (&qf)[2][NKS], float sl2, float neg, float (&lsum)[2],
                                 const bf16x8* lds, int lane) {
  float y[2][2], e[2][2], s[2][2] = {{0.0f, 0.0f}, {0.0f, 0.0f}};
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    y[0][i] = __builtin_fmaf(in[0][i], sl2, neg);
    pin(y[0][i]);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int g = 0; g < 2 * NKS; ++g) {
    const int ks = g >> 1, cb = g & 1, b = g & 1;
    if (cb == 0) pin(f[ks]);
    pin(qf[cb][ks]);
    o[cb] = mma(f[ks], qf[cb][ks], ks ? o[cb] : floatx16{});
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      e[b][i] = __builtin_amdgcn_exp2f(y[b][i]);
      pin(e[b][i]);
    }
    if (g > 0) {
#pragma unroll
      for (int i = 0; i < 2; ++i) s[cb ^ 1][i] += e[b ^ 1][i];
      pin(s[cb ^ 1][0]);
      pin(s[cb ^ 1][1]);
    }
    if (g + 1 < 2 * NKS) {
      const int ncb = (g + 1) & 1, nks = (g + 1) >> 1;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        y[b ^ 1][i] = __builtin_fmaf(in[ncb][nks * 2 + i], sl2, neg);
        pin(y[b ^ 1][i]);
      }
    }
    if (LDS && cb == 1) f[ks] = lds[(ks * 64 + lane) & 511];  // next phase's fragment of this k-step
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) s[1][i] += e[1][i];
  lsum[0] += s[0][0] + s[0][1];
  lsum[1] += s[1][0] + s[1][1];
}

template <bool LDS, bool BAR = false>
__global__ __launch_bounds__(256, 2) void probe_mix(int iters, float* out, int flag) {
  __shared__ bf16x8 tile[512];  // 8 KB of key fragments
  const int lane = threadIdx.x & 63;
  if (LDS) {
    for (int i = threadIdx.x; i < 512; i += blockDim.x) tile[i] = frag_of(i);
    __syncthreads();
  }
  bf16x8 f[NKS], qf[2][NKS];
#pragma unroll
  for (int k = 0; k < NKS; ++k) {
    f[k] = frag_of(threadIdx.x + k);
    qf[0][k] = frag_of(threadIdx.x + 2 * k);
    qf[1][k] = frag_of(threadIdx.x + 3 * k);
  }
  floatx16 acc0[2] = {}, acc1[2] = {};
  float lsum[2] = {0.0f, 0.0f};
  const float sl2 = 0.1275f, neg = -1.0f;
  for (int it = 0; it < iters; ++it) {
    mix_phase<LDS>(acc0, acc1, f, qf, sl2, neg, lsum, tile, lane);
    if (BAR) __syncthreads();  // the passes hand each tile to the workgroup's waves with one barrier
    mix_phase<LDS>(acc1, acc0, f, qf, sl2, neg, lsum, tile, lane);
  }
  if (flag) out[blockIdx.x * blockDim.x + threadIdx.x] = lsum[0] + lsum[1] + acc0[0][0] + acc1[1][1];
}

// v_max_f32 / v_max3_f32 written out, as the Gram pass writes them.
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

// One phase of the Gram mix: MFMAs into `o` (two register row blocks x NKS
// k-steps against one tile fragment per k-step) interleaved with the
// cosines and maxima of the products in `in`, as the Gram pass schedules it.
__device__ inline void gram_phase(floatx16 (&o)[2], bf16x8 (&a)[2][NKS], const bf16x8* lds, int lane,
                                  const floatx16 (&in)[2], float invj, float (&iv)[2][16], float (&rmax)[2][16],
                                  float& cm) {
  constexpr int NG = 2 * NKS;
  constexpr int PER = 32 / NG;
  static_assert(PER == 2, "two products per MFMA");
  bf16x8 f[NKS];
  f[0] = lds[lane & 511];
  f[1] = lds[(64 + lane) & 511];
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int ks = g >> 1, rb = g & 1;
    if (rb == 0 && ks + 2 < NKS) f[ks + 2] = lds[((ks + 2) * 64 + lane) & 511];
    pin(a[rb][ks]);
    o[rb] = mma(a[rb][ks], f[ks], ks ? o[rb] : floatx16{});
    float c[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = g * PER + i, erb = e >> 4, r = e & 15;
      c[i] = in[erb][r] * invj * iv[erb][r];
      rmax[erb][r] = vmax(rmax[erb][r], c[i]);
      pin(rmax[erb][r]);
    }
    cm = vmax3(cm, c[0], c[1]);
    pin(cm);
    __builtin_amdgcn_sched_barrier(0);
  }
}

__global__ __launch_bounds__(256, 2) void probe_gram(int iters, float* out, int flag) {
  __shared__ bf16x8 tile[512];  // 8 KB of tile-row fragments
  const int lane = threadIdx.x & 63;
  for (int i = threadIdx.x; i < 512; i += blockDim.x) tile[i] = frag_of(i);
  __syncthreads();
  bf16x8 a[2][NKS];
  float iv[2][16], rmax[2][16];
#pragma unroll
  for (int k = 0; k < NKS; ++k) {
    a[0][k] = frag_of(threadIdx.x + 2 * k);
    a[1][k] = frag_of(threadIdx.x + 3 * k);
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    iv[0][r] = 1.0f + 0.01f * (float)r;
    iv[1][r] = 1.0f - 0.01f * (float)r;
    rmax[0][r] = rmax[1][r] = -1.0f;
  }
  floatx16 acc0[2] = {}, acc1[2] = {};
  const float invj = 0.9f + 0.001f * (float)lane;
  float cm = -1.0f, cms = 0.0f;
  for (int it = 0; it < iters; ++it) {
    gram_phase(acc1, a, tile, lane, acc0, invj, iv, rmax, cm);
    cms += cm;
    __syncthreads();  // the pass hands each tile to the workgroup's waves with one barrier
    gram_phase(acc0, a, tile, lane, acc1, invj, iv, rmax, cm);
    cms += cm;
  }
  float t = cms + acc0[0][0] + acc1[1][1];
#pragma unroll
  for (int r = 0; r < 16; ++r) t += rmax[0][r] + rmax[1][r];
  if (flag) out[blockIdx.x * blockDim.x + threadIdx.x] = t;
}

}  // namespace

extern "C" {

// Launch probe `kind` (0 MFMA, 1 exp2, 2 mix, 3 mix with LDS fragments, 4 the
// same with a barrier per tile, 5 the Gram mix) on
// `blocks` workgroups of 256 threads for `iters` iterations on `stream`.
// Work per launch, per wave: kind 0: 4 * iters MFMAs; kind 1: 16 * iters
// exp2; kinds 2-4: 32 * iters MFMAs and 64 * iters exp2; kind 5: 32 * iters
// MFMAs and 64 * iters cosines.  `out` receives nothing unless `flag` is
// set.  Returns a hipError_t.
int omnimem_probe_run(int kind, int blocks, int iters, float* out, int flag, hipStream_t stream) {
  if (blocks < 1 || iters < 1 || kind < 0 || kind > 5) return (int)hipErrorInvalidValue;
  switch (kind) {
    case 0: probe_mfma<<<blocks, 256, 0, stream>>>(iters, out, flag); break;
    case 1: probe_exp<<<blocks, 256, 0, stream>>>(iters, out, flag); break;
    case 2: probe_mix<false><<<blocks, 256, 0, stream>>>(iters, out, flag); break;
    case 3: probe_mix<true><<<blocks, 256, 0, stream>>>(iters, out, flag); break;
    case 4: probe_mix<true, true><<<blocks, 256, 0, stream>>>(iters, out, flag); break;
    default: probe_gram<<<blocks, 256, 0, stream>>>(iters, out, flag); break;
  }
  return (int)hipGetLastError();
}

}  // extern "C"
