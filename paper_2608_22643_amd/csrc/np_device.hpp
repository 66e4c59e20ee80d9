// np_device.hpp -- device-side building blocks for gfx950 (64-wide waves):
// element types moved as 16-byte vectors, dot products on the packed dot
// instructions, wave reductions, workgroup scans, the sticky error word and
// the workgroup k-selection primitive shared by top-k and victim selection.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "np_internal.hpp"

namespace np {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf162_t __attribute__((ext_vector_type(2)));

constexpr int WAVE = 64;

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// 16-byte load with the nontemporal hint (data streamed once)
__device__ inline uint4 load_nt(const uint4* p) {
  const u32x4_t v = __builtin_nontemporal_load((const u32x4_t*)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// A 16-byte store with the nontemporal hint (written records go to memory
// without lingering as dirty lines that later kernels would have to flush).
__device__ inline void store_nt(uint4* p, uint4 x) {
  u32x4_t v;
  v.x = x.x;
  v.y = x.y;
  v.z = x.z;
  v.w = x.w;
  __builtin_nontemporal_store(v, (u32x4_t*)p);
}

// Buffer loads: a 128-bit resource (base, size) held in scalar registers plus
// a 32-bit per-lane byte offset, so no 64-bit address arithmetic per lane.
// The hardware range-checks the per-lane offset: an offset at or past the
// size returns zeros without a memory access (BUF_OOB below).
constexpr uint32_t BUF_OOB = 0x7FFFFFFFu;
constexpr int BUF_RSRC_WORD3 = 0x00020000;  // raw 32-bit buffer, gfx9 family

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, (int)bytes, BUF_RSRC_WORD3);
}

__device__ inline uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// The same with the nontemporal hint: weight records streamed once per use,
// which the caches need not keep (measured 3-8% faster for the MLP streams).
constexpr int CPOL_NT = 2;
__device__ inline uint4 buf_load16_nt(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, CPOL_NT);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Cache policy "sc1" on gfx950: agent (device) scope.  A store with it is
// written through to the point of coherence shared by all XCDs, and a load
// with it reads that point, so data passes between workgroups on different
// XCDs inside one kernel without an L2 write-back or invalidate.
constexpr int CPOL_SC1 = 16;

__device__ inline float4 buf_load16_agent(__amdgpu_buffer_rsrc_t r, uint32_t voff) {
  const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, 0, CPOL_SC1);
  return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z),
                     __uint_as_float(v.w));
}

// A 16-byte store with the nontemporal hint: data the next kernel reads once
// (the MLP's partial sums) need not displace other lines on the way.
__device__ inline void buf_store16_nt(__amdgpu_buffer_rsrc_t r, uint32_t voff, float4 f) {
  u32x4_t v;
  v.x = __float_as_uint(f.x);
  v.y = __float_as_uint(f.y);
  v.z = __float_as_uint(f.z);
  v.w = __float_as_uint(f.w);
  __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)voff, 0, CPOL_NT);
}

__device__ inline void buf_store16_agent(__amdgpu_buffer_rsrc_t r, uint32_t voff, float4 f) {
  u32x4_t v;
  v.x = __float_as_uint(f.x);
  v.y = __float_as_uint(f.y);
  v.z = __float_as_uint(f.z);
  v.w = __float_as_uint(f.w);
  __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)voff, 0, CPOL_SC1);
}

// ---------------------------------------------------------------------------
// element types.  A 16-byte vector (uint4) holds V elements.
// dot(w, x, acc): acc + sum_e w[e] * x[e] in fp32 (packed dot instructions
// for 16-bit types: products are exact in fp32).
// axpy(acc, a, w): acc[e] += a * float(w[e]).
// ---------------------------------------------------------------------------
struct TF32 {
  static constexpr int V = 4;
  static constexpr int dtype = NP_F32;
  __device__ static inline float dot(uint4 w, uint4 x, float acc) {
    acc = __builtin_fmaf(__uint_as_float(w.x), __uint_as_float(x.x), acc);
    acc = __builtin_fmaf(__uint_as_float(w.y), __uint_as_float(x.y), acc);
    acc = __builtin_fmaf(__uint_as_float(w.z), __uint_as_float(x.z), acc);
    acc = __builtin_fmaf(__uint_as_float(w.w), __uint_as_float(x.w), acc);
    return acc;
  }
  __device__ static inline void axpy(float* acc, float a, uint4 w) {
    acc[0] = __builtin_fmaf(a, __uint_as_float(w.x), acc[0]);
    acc[1] = __builtin_fmaf(a, __uint_as_float(w.y), acc[1]);
    acc[2] = __builtin_fmaf(a, __uint_as_float(w.z), acc[2]);
    acc[3] = __builtin_fmaf(a, __uint_as_float(w.w), acc[3]);
  }
  __device__ static inline void unpack(uint4 w, float* f) {
    f[0] = __uint_as_float(w.x);
    f[1] = __uint_as_float(w.y);
    f[2] = __uint_as_float(w.z);
    f[3] = __uint_as_float(w.w);
  }
  __device__ static inline uint32_t from_f32(float f) { return __float_as_uint(f); }
};

__device__ inline half2_t as_h2(uint32_t u) { return __builtin_bit_cast(half2_t, u); }
__device__ inline bf162_t as_b2(uint32_t u) { return __builtin_bit_cast(bf162_t, u); }

struct TF16 {
  static constexpr int V = 8;
  static constexpr int dtype = NP_F16;
  __device__ static inline float dot(uint4 w, uint4 x, float acc) {
    acc = __builtin_amdgcn_fdot2(as_h2(w.x), as_h2(x.x), acc, false);
    acc = __builtin_amdgcn_fdot2(as_h2(w.y), as_h2(x.y), acc, false);
    acc = __builtin_amdgcn_fdot2(as_h2(w.z), as_h2(x.z), acc, false);
    acc = __builtin_amdgcn_fdot2(as_h2(w.w), as_h2(x.w), acc, false);
    return acc;
  }
  __device__ static inline float lo(uint32_t u) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(u & 0xFFFFu));
  }
  __device__ static inline float hi(uint32_t u) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(u >> 16));
  }
  __device__ static inline void unpack(uint4 w, float* f) {
    f[0] = lo(w.x);
    f[1] = hi(w.x);
    f[2] = lo(w.y);
    f[3] = hi(w.y);
    f[4] = lo(w.z);
    f[5] = hi(w.z);
    f[6] = lo(w.w);
    f[7] = hi(w.w);
  }
  __device__ static inline void axpy(float* acc, float a, uint4 w) {
    acc[0] = __builtin_fmaf(a, lo(w.x), acc[0]);
    acc[1] = __builtin_fmaf(a, hi(w.x), acc[1]);
    acc[2] = __builtin_fmaf(a, lo(w.y), acc[2]);
    acc[3] = __builtin_fmaf(a, hi(w.y), acc[3]);
    acc[4] = __builtin_fmaf(a, lo(w.z), acc[4]);
    acc[5] = __builtin_fmaf(a, hi(w.z), acc[5]);
    acc[6] = __builtin_fmaf(a, lo(w.w), acc[6]);
    acc[7] = __builtin_fmaf(a, hi(w.w), acc[7]);
  }
  // fp32 -> binary16, round to nearest even (the hardware conversion)
  __device__ static inline uint32_t from_f32(float f) {
    return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)f);
  }
};

struct TBF16 {
  static constexpr int V = 8;
  static constexpr int dtype = NP_BF16;
  __device__ static inline float dot(uint4 w, uint4 x, float acc) {
    acc = __builtin_amdgcn_fdot2_f32_bf16(as_b2(w.x), as_b2(x.x), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(as_b2(w.y), as_b2(x.y), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(as_b2(w.z), as_b2(x.z), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(as_b2(w.w), as_b2(x.w), acc, false);
    return acc;
  }
  // bf16 -> fp32 is exact: the bf16 bits are the top half of the fp32 bits
  __device__ static inline float lo(uint32_t u) { return __uint_as_float(u << 16); }
  __device__ static inline float hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }
  __device__ static inline void unpack(uint4 w, float* f) {
    f[0] = lo(w.x);
    f[1] = hi(w.x);
    f[2] = lo(w.y);
    f[3] = hi(w.y);
    f[4] = lo(w.z);
    f[5] = hi(w.z);
    f[6] = lo(w.w);
    f[7] = hi(w.w);
  }
  __device__ static inline void axpy(float* acc, float a, uint4 w) {
    acc[0] = __builtin_fmaf(a, lo(w.x), acc[0]);
    acc[1] = __builtin_fmaf(a, hi(w.x), acc[1]);
    acc[2] = __builtin_fmaf(a, lo(w.y), acc[2]);
    acc[3] = __builtin_fmaf(a, hi(w.y), acc[3]);
    acc[4] = __builtin_fmaf(a, lo(w.z), acc[4]);
    acc[5] = __builtin_fmaf(a, hi(w.z), acc[5]);
    acc[6] = __builtin_fmaf(a, lo(w.w), acc[6]);
    acc[7] = __builtin_fmaf(a, hi(w.w), acc[7]);
  }
  // fp32 -> bfloat16, round to nearest even; NaN stays a quiet NaN
  __device__ static inline uint32_t from_f32(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (u >> 16) | 0x40u;
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
  }
};

// ---------------------------------------------------------------------------
// matrix cores: one "step" of a 16 x 16 fp32 tile over 4*V reduction elements
// (one v_mfma_f32_16x16x32 for 16-bit types, four v_mfma_f32_16x16x4f32 for
// fp32).  Lane l holds row l%16 of the A operand and column l%16 of the B
// operand, each as the V consecutive elements starting at V*(l/16) of the
// step; the accumulator's register i of lane l is output row 4*(l/16) + i,
// column l%16.
// ---------------------------------------------------------------------------
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <class T>
__device__ inline f32x4 mfma_step(uint4 a, uint4 b, f32x4 c) {
  if constexpr (T::dtype == NP_F16) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  } else if constexpr (T::dtype == NP_BF16) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  } else {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0,
                                                0);
  }
}

// ---------------------------------------------------------------------------
// wave / workgroup reductions and scans
// ---------------------------------------------------------------------------
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, WAVE);
  return v;
}

// Sum over aligned groups of G lanes (G a power of two <= 64); every lane of
// the group receives the group sum.  Fixed order: deterministic.
template <int G>
__device__ inline float group_sum(float v) {
#pragma unroll
  for (int off = G / 2; off >= 1; off >>= 1) v += __shfl_xor(v, off, WAVE);
  return v;
}

// Reduce-scatter of N values (N a power of two, 2 <= N <= 64) over a wave:
// on entry every lane holds v[0..N-1]; on return lane l holds in v[0] the
// wave sum of value l / (64/N) (every lane of that group of 64/N lanes holds
// it).  Each halving step sends the half a lane gives up to its partner, so
// the N sums cost N - 1 + log2(64/N) shuffles instead of N * 6.  Element
// indices are template constants throughout, so every access is static and
// each choice between two halves is one select.
template <int I, int HALF, int M>
struct RsStep {
  template <int N>
  __device__ static inline void run(float (&v)[N], bool hi) {
    const float send = hi ? v[I] : v[I + HALF];
    const float keep = hi ? v[I + HALF] : v[I];
    v[I] = keep + __shfl_xor(send, M, WAVE);
    RsStep<I + 1, HALF, M>::run(v, hi);
  }
};
template <int HALF, int M>
struct RsStep<HALF, HALF, M> {
  template <int N>
  __device__ static inline void run(float (&)[N], bool) {}
};

template <int CNT, int M>
struct RsLevel {  // CNT values left, partner distance M
  template <int N>
  __device__ static inline void run(float (&v)[N], int lane) {
    RsStep<0, CNT / 2, M>::run(v, (lane & M) != 0);
    RsLevel<CNT / 2, M / 2>::run(v, lane);
  }
};
template <int M>
struct RsLevel<1, M> {  // one value left: sum it over the remaining lanes
  template <int N>
  __device__ static inline void run(float (&v)[N], int) {
#pragma unroll
    for (int m = M; m >= 1; m >>= 1) v[0] += __shfl_xor(v[0], m, WAVE);
  }
};

template <int N>
__device__ inline void wave_reduce_scatter(float (&v)[N]) {
  static_assert(N >= 2 && N <= WAVE && (N & (N - 1)) == 0, "N: power of two in [2, 64]");
  RsLevel<N, WAVE / 2>::run(v, (int)(threadIdx.x & (WAVE - 1)));
}

__device__ inline uint32_t wave_incl_scan(uint32_t v) {
  const int lane = threadIdx.x & (WAVE - 1);
#pragma unroll
  for (int off = 1; off < WAVE; off <<= 1) {
    uint32_t y = __shfl_up(v, off, WAVE);
    if (lane >= off) v += y;
  }
  return v;
}

// Exclusive prefix sum over the NT threads of a workgroup, in thread order.
// lds must hold NT/64 + 1 uint32.  Returns the exclusive value; *total gets
// the sum.  Contains barriers: every thread must call it.
template <int NT>
__device__ inline uint32_t block_excl_scan(uint32_t v, uint32_t* lds, uint32_t* total) {
  constexpr int NW = NT / WAVE;
  const int lane = threadIdx.x & (WAVE - 1), w = threadIdx.x / WAVE;
  uint32_t incl = wave_incl_scan(v);
  if (lane == WAVE - 1) lds[w] = incl;
  __syncthreads();
  if (w == 0) {
    uint32_t t = lane < NW ? lds[lane] : 0u;
    uint32_t ti = wave_incl_scan(t);
    if (lane < NW) lds[lane] = ti - t;
    if (lane == NW - 1) lds[NW] = ti;
  }
  __syncthreads();
  uint32_t res = lds[w] + incl - v;
  *total = lds[NW];
  __syncthreads();
  return res;
}

// ---------------------------------------------------------------------------
// gated activation of an MLP neuron: a = act(g, u), ReLU-gated max(g, 0) u or
// SwiGLU SiLU(g) u with SiLU(g) = g / (1 + e^-g) (HIP's expf, IEEE divide)
// ---------------------------------------------------------------------------
__device__ inline float gated(int act, float g, float u) {
  if (act == NP_ACT_SWIGLU) return g / (1.f + expf(-g)) * u;
  return fmaxf(g, 0.f) * u;
}

// ---------------------------------------------------------------------------
// sticky device error word
// ---------------------------------------------------------------------------
__device__ inline void raise_error(void* ws, int bits) {
  atomicOr((int*)((char*)ws + WS_ERR), bits);
}

// ---------------------------------------------------------------------------
// k-selection over one workgroup (NT threads).  Each thread owns WPT
// consecutive 32-id words (thread t: words t*WPT .. t*WPT+WPT-1), and key[w][b]
// is the 32-bit unsigned key of id 32*(t*WPT+w)+b.  Selects the `kk` largest
// keys; ties at the kk-th key go to the smaller ids.  On return sel[w] holds
// the selected bits of each owned word.
//
// Key 0 marks ids that are outside the range or not candidates; such keys
// are taken only when fewer than kk keys are nonzero (then in id order).
// Radix select from the top over the nonzero keys on an LDS histogram of up
// to 12 bits per pass, starting at the highest bit in which the nonzero keys
// differ: fp32 score keys need at most three passes, least-recently-used
// keys (a narrow range of token indices under a common prefix) usually one,
// and no pass piles every key onto one histogram bin.  Once at most
// SEL_SMALL_CAND keys remain under the prefix, or at most 8 bits, passes
// take 8 bits and wave 0 alone finds the bin among 256.  A pass whose bin holds exactly the keys
// still needed ends the search: every key of the bin is selected, so the
// kk-th key is the bin's smallest, found by one reduction instead of further
// passes (fp32 scores: usually after the second pass).  Then an ordered scan
// of the ties.  hist: 4096 uint32 of LDS; scan: 3*NT/64 + 1 uint32; res: 4
// uint32.
// ---------------------------------------------------------------------------
constexpr uint32_t SEL_SMALL_CAND = 1024;  // at most this many keys left: 8-bit passes

template <int NT, int WPT>
__device__ inline void block_select_largest(const uint32_t (&key)[WPT][32], uint32_t kk,
                                            uint32_t (&sel)[WPT], uint32_t* hist,
                                            uint32_t* scan, uint32_t* res) {
  constexpr int NW = NT / WAVE;
  const int tid = threadIdx.x, lane = tid & (WAVE - 1), w = tid / WAVE;
  // count, max and min of the nonzero keys
  uint32_t nz = 0, kmax = 0, kmin = 0xFFFFFFFFu;
#pragma unroll
  for (int i = 0; i < WPT; ++i)
#pragma unroll
    for (int b = 0; b < 32; ++b) {
      const uint32_t kv = key[i][b];
      nz += kv != 0u;
      kmax = kv > kmax ? kv : kmax;
      kmin = (kv != 0u && kv < kmin) ? kv : kmin;
    }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    nz += __shfl_xor(nz, off, WAVE);
    const uint32_t a = __shfl_xor(kmax, off, WAVE), c = __shfl_xor(kmin, off, WAVE);
    kmax = a > kmax ? a : kmax;
    kmin = c < kmin ? c : kmin;
  }
  if (lane == 0) {
    scan[w] = nz;
    scan[NW + w] = kmax;
    scan[2 * NW + w] = kmin;
  }
  __syncthreads();
  nz = 0;
  kmax = 0;
  kmin = 0xFFFFFFFFu;
  for (int i = 0; i < NW; ++i) {
    nz += scan[i];
    kmax = scan[NW + i] > kmax ? scan[NW + i] : kmax;
    kmin = scan[2 * NW + i] < kmin ? scan[2 * NW + i] : kmin;
  }
  __syncthreads();  // scan is reused below

  uint32_t prefix, rem;
  if (kk >= nz) {  // every nonzero key, then the first kk - nz zero keys
    prefix = 0u;
    rem = kk - nz;
  } else {  // the kk-th largest key is nonzero: zero keys take no part
    const uint32_t diff = kmax ^ kmin;
    int hi = diff ? 31 - __builtin_clz(diff) : -1;  // highest differing bit
    const uint32_t low = hi >= 0 ? (uint32_t)((2ull << hi) - 1ull) : 0u;
    prefix = kmax & ~low;  // bits above hi are common to all nonzero keys
    uint32_t pmask = ~low;
    rem = kk;
    uint32_t ncand = nz;  // keys under the prefix so far
    while (hi >= 0) {  // uniform: every thread runs the same passes
      // few keys left: an 8-bit digit, whose 256 bins wave 0 scans alone;
      // otherwise 12 bits and a workgroup scan over the 4096 bins
      const bool small = ncand <= SEL_SMALL_CAND || hi + 1 <= 8;
      const int maxbits = small ? 8 : 12;
      const int nbits = hi + 1 < maxbits ? hi + 1 : maxbits;
      const int shift = hi + 1 - nbits;
      const uint32_t nb = 1u << nbits;
      for (uint32_t i = tid; i < nb; i += NT) hist[i] = 0;
      __syncthreads();
#pragma unroll
      for (int i = 0; i < WPT; ++i)
#pragma unroll
        for (int b = 0; b < 32; ++b) {
          const uint32_t kv = key[i][b];
          if (kv != 0u && (kv & pmask) == prefix) atomicAdd(&hist[(kv >> shift) & (nb - 1)], 1u);
        }
      __syncthreads();
      if (small) {
        if (w == 0) {  // lane L: bins [nb - 4(L+1), nb - 4L), from the top
          uint32_t local = 0;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int bin = (int)nb - 4 * lane - 1 - i;
            if (bin >= 0) local += hist[bin];
          }
          const uint32_t incl = wave_incl_scan(local), above = incl - local;
          if (above < rem && incl >= rem) {
            uint32_t c = above;
            for (int i = 0; i < 4; ++i) {
              const int bin = (int)nb - 4 * lane - 1 - i;
              const uint32_t h = hist[bin];
              if (c + h >= rem) {
                res[0] = (uint32_t)bin;
                res[1] = rem - c;
                res[2] = h == rem - c;  // the whole bin is needed
                res[3] = h;
                break;
              }
              c += h;
            }
          }
        }
      } else {
        // thread t owns bins [nb - (t+1)*bpt, nb - t*bpt): counting from the top
        const uint32_t bpt = nb >= (uint32_t)NT ? nb / NT : 1u;
        const bool owner = (uint32_t)tid * bpt < nb;
        const uint32_t hi_bin = nb - (uint32_t)tid * bpt;  // exclusive
        uint32_t local = 0;
        if (owner)
          for (uint32_t i = 0; i < bpt; ++i) local += hist[hi_bin - 1 - i];
        uint32_t tot;
        const uint32_t above = block_excl_scan<NT>(local, scan, &tot);
        if (owner && above < rem && above + local >= rem) {
          uint32_t c = above;
          for (uint32_t i = 0; i < bpt; ++i) {
            const uint32_t bin = hi_bin - 1 - i;
            if (c + hist[bin] >= rem) {
              res[0] = bin;
              res[1] = rem - c;
              res[2] = hist[bin] == rem - c;  // the whole bin is needed
              res[3] = hist[bin];
              break;
            }
            c += hist[bin];
          }
        }
      }
      __syncthreads();
      prefix |= res[0] << shift;
      pmask |= (nb - 1) << shift;
      rem = res[1];
      ncand = res[3];
      hi = shift - 1;
      const bool whole = res[2] != 0u && hi >= 0;
      __syncthreads();
      if (whole) {
        // every key of the bin is taken: the kk-th largest is its smallest
        // key, and every key equal to it is taken too (rem: no limit)
        uint32_t kmn = 0xFFFFFFFFu;
#pragma unroll
        for (int i = 0; i < WPT; ++i)
#pragma unroll
          for (int b = 0; b < 32; ++b) {
            const uint32_t kv = key[i][b];
            if (kv != 0u && (kv & pmask) == prefix && kv < kmn) kmn = kv;
          }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
          const uint32_t c = __shfl_xor(kmn, off, WAVE);
          kmn = c < kmn ? c : kmn;
        }
        if (lane == 0) scan[w] = kmn;
        __syncthreads();
        kmn = scan[0];
        for (int i = 1; i < NW; ++i) kmn = scan[i] < kmn ? scan[i] : kmn;
        __syncthreads();  // scan is reused below
        prefix = kmn;
        rem = 0xFFFFFFFFu;
        break;
      }
    }
  }
  // prefix is the kk-th largest key; take all larger keys and the first `rem`
  // equal keys in id order.
  uint32_t eqm[WPT], neq = 0;
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    uint32_t gt = 0, eq = 0;
#pragma unroll
    for (int b = 0; b < 32; ++b) {
      gt |= (key[i][b] > prefix ? 1u : 0u) << b;
      eq |= (key[i][b] == prefix ? 1u : 0u) << b;
    }
    sel[i] = gt;
    eqm[i] = eq;
    neq += __builtin_popcount(eq);
  }
  uint32_t tot;
  uint32_t before = block_excl_scan<NT>(neq, scan, &tot);
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    uint32_t e = eqm[i];
    while (e && before < rem) {
      uint32_t lowbit = e & (0u - e);
      sel[i] |= lowbit;
      e ^= lowbit;
      ++before;
    }
  }
}

}  // namespace np
