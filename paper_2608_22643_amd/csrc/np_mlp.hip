// np_mlp.hip -- sparse ReLU-gated MLP of one downstream layer over its
// resident active rows (Sec. 3.4: the slot map locates each active row, row
// order is irrelevant; Sec. 3.3: the down projection's output stays dense):
//     y = sum_j max(gate_j . x, 0) * (up_j . x) * downT_j
// Row j is one resident record [gate | up | downT] (3d contiguous elements),
// so the kernel streams whole 24 KiB records at 7B shape: HBM-bound.
//
// Work split (one launch per layer):
//   * a workgroup of 8 waves owns a contiguous range of the active list;
//   * a row is handled by P waves (P = 1 up to d = 4096 for 16-bit types),
//     each covering a contiguous part of d; lane i reads 16-byte vectors
//     i, i+64, ... of the part, so every wave instruction reads 1 KiB of
//     contiguous memory; all gate/up/downT loads of a row are issued before
//     any arithmetic;
//   * g and u are wave sums (plus an LDS exchange when P > 1); each wave
//     accumulates a * downT into fp32 registers;
//   * the 8 waves' partial y meet in an LDS tree (fixed order), each
//     workgroup writes one fp32 partial of y to the workspace;
//   * the last n_red workgroups to finish (an arrival ticket) wait for the
//     rest, then each sums the partials of d/n_red columns in workgroup
//     order and writes y rounded once to the activation type.  The waits are
//     bounded: every waiting workgroup is among the last to arrive, so the
//     ones it waits for are already resident or free to be scheduled.
#include <stdlib.h>

#include <algorithm>

#include "np_device.hpp"

namespace np {

constexpr int MLP_NW = 8;
constexpr int MLP_NT = MLP_NW * WAVE;
constexpr uint32_t MLP_SPIN_LIMIT = 1u << 22;

struct MlpArgs {
  const uint4* res_layer;  // first record of the layer in the resident buffer
  const int32_t* slots;    // active_slots of the layer
  const uint4* x;
  void* y;
  float* partials;         // [n_wg][d]
  uint32_t* arrive;
  uint32_t* done;
  void* ws;
  int n_active, C, NV, NVP, rows_per_wg, n_wg, n_red, d;
};

template <class T>
__device__ inline void store_y4(void* y, int col, float4 v) {
  if constexpr (T::dtype == NP_F32) {
    *(float4*)((float*)y + col) = v;
  } else {
    uint2 o;
    o.x = T::from_f32(v.x) | (T::from_f32(v.y) << 16);
    o.y = T::from_f32(v.z) | (T::from_f32(v.w) << 16);
    *(uint2*)((uint16_t*)y + col) = o;
  }
}

template <class T, int CPL, int P>
__global__ __launch_bounds__(MLP_NT) void sparse_mlp_kernel(MlpArgs a) {
  constexpr int V = T::V;
  constexpr int Q = MLP_NW / P;  // waves sharing one part of d
  extern __shared__ float4 smem_f4[];
  float* red = (float*)smem_f4;
  __shared__ float gu[MLP_NW][2];
  __shared__ uint32_t s_ticket;

  const int tid = threadIdx.x, lane = tid & (WAVE - 1), w = tid / WAVE;
  const int q = w / P, p = w % P;
  const int b = blockIdx.x;
  const int row_begin = b * a.rows_per_wg;
  const int row_end = min(row_begin + a.rows_per_wg, a.n_active);
  const int part_v0 = p * a.NVP;
  const int part_len = min(a.NVP, a.NV - part_v0);

  uint4 xr[CPL];
  bool vok[CPL];
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int off = lane + WAVE * c;
    vok[c] = off < part_len;
    xr[c] = vok[c] ? a.x[part_v0 + off] : make_uint4(0u, 0u, 0u, 0u);
  }
  float yacc[CPL][V];
#pragma unroll
  for (int c = 0; c < CPL; ++c)
#pragma unroll
    for (int e = 0; e < V; ++e) yacc[c][e] = 0.f;

  for (int r0 = row_begin; r0 < row_end; r0 += Q) {
    const int row = r0 + q;
    bool valid = row < row_end;
    int slot = -1;
    if (valid) {
      slot = a.slots[row];
      if (slot < 0 || slot >= a.C) {
        if (lane == 0 && p == 0) raise_error(a.ws, NP_DEVERR_NOT_RESIDENT);
        valid = false;
      }
    }
    const uint4* rec = a.res_layer + (size_t)(valid ? slot : 0) * 3 * a.NV + part_v0;
    uint4 gw[CPL], uw[CPL], dw[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      const int off = lane + WAVE * c;
      if (valid && vok[c]) {
        gw[c] = load_nt(rec + off);
        uw[c] = load_nt(rec + a.NV + off);
        dw[c] = load_nt(rec + 2 * a.NV + off);
      } else {
        gw[c] = uw[c] = dw[c] = make_uint4(0u, 0u, 0u, 0u);
      }
    }
    float g = 0.f, u = 0.f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      g = T::dot(gw[c], xr[c], g);
      u = T::dot(uw[c], xr[c], u);
    }
    g = wave_sum(g);
    u = wave_sum(u);
    if constexpr (P > 1) {
      if (lane == 0) {
        gu[w][0] = g;
        gu[w][1] = u;
      }
      __syncthreads();
      g = 0.f;
      u = 0.f;
#pragma unroll
      for (int pp = 0; pp < P; ++pp) {
        g += gu[q * P + pp][0];
        u += gu[q * P + pp][1];
      }
      __syncthreads();
    }
    if (valid) {
      const float act = fmaxf(g, 0.f) * u;
#pragma unroll
      for (int c = 0; c < CPL; ++c)
        if (vok[c]) T::axpy(yacc[c], act, dw[c]);
    }
  }

  // partial sums of the Q waves of each part meet in an LDS tree
  const int part_floats = a.NVP * V;
#pragma unroll
  for (int s = Q / 2; s >= 1; s /= 2) {
    if (q >= s && q < 2 * s) {
      float* dst = red + (size_t)((q - s) * P + p) * part_floats;
#pragma unroll
      for (int c = 0; c < CPL; ++c)
        if (vok[c]) {
          float4* d4 = (float4*)(dst + (lane + WAVE * c) * V);
#pragma unroll
          for (int e = 0; e < V; e += 4)
            d4[e / 4] = make_float4(yacc[c][e], yacc[c][e + 1], yacc[c][e + 2], yacc[c][e + 3]);
        }
    }
    __syncthreads();
    if (q < s) {
      const float* src = red + (size_t)(q * P + p) * part_floats;
#pragma unroll
      for (int c = 0; c < CPL; ++c)
        if (vok[c]) {
          const float4* s4 = (const float4*)(src + (lane + WAVE * c) * V);
#pragma unroll
          for (int e = 0; e < V; e += 4) {
            const float4 t = s4[e / 4];
            yacc[c][e] += t.x;
            yacc[c][e + 1] += t.y;
            yacc[c][e + 2] += t.z;
            yacc[c][e + 3] += t.w;
          }
        }
    }
    __syncthreads();
  }
  if (q == 0) {
    float* dstp = a.partials + (size_t)b * a.d + (size_t)part_v0 * V;
#pragma unroll
    for (int c = 0; c < CPL; ++c)
      if (vok[c]) {
        float4* d4 = (float4*)(dstp + (lane + WAVE * c) * V);
#pragma unroll
        for (int e = 0; e < V; e += 4)
          d4[e / 4] = make_float4(yacc[c][e], yacc[c][e + 1], yacc[c][e + 2], yacc[c][e + 3]);
      }
  }

  // arrival: release this workgroup's partial, take a ticket
  __threadfence();
  __syncthreads();
  if (tid == 0) s_ticket = atomicAdd(a.arrive, 1u);
  __syncthreads();
  const uint32_t ticket = s_ticket;
  if (ticket < (uint32_t)(a.n_wg - a.n_red)) return;

  // one of the last n_red arrivals: wait for the others, then reduce a slice
  const int ri = (int)ticket - (a.n_wg - a.n_red);
  if (tid == 0) {
    uint32_t it = 0;
    while (__hip_atomic_load(a.arrive, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) <
           (uint32_t)a.n_wg) {
      __builtin_amdgcn_s_sleep(1);
      if (++it > MLP_SPIN_LIMIT) {
        raise_error(a.ws, NP_DEVERR_SPIN_LIMIT);
        break;
      }
    }
  }
  __syncthreads();
  __threadfence();

  const int CR = a.d / a.n_red;  // columns of this reducer, multiple of 4
  const int G4 = CR / 4;
  const int TPC = G4 < MLP_NT ? G4 : MLP_NT;
  const int RG = MLP_NT / TPC;
  float4* red4 = smem_f4;
  for (int cg0 = 0; cg0 < G4; cg0 += TPC) {
    const int cg = cg0 + tid % TPC, rg = tid / TPC;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (cg < G4 && rg < RG) {
      const int col = ri * CR + 4 * cg;
      for (int bb = rg; bb < a.n_wg; bb += RG) {
        const float4 t = *(const float4*)(a.partials + (size_t)bb * a.d + col);
        acc.x += t.x;
        acc.y += t.y;
        acc.z += t.z;
        acc.w += t.w;
      }
    }
    if (rg < RG) red4[rg * TPC + tid % TPC] = acc;
    __syncthreads();
    if (tid < TPC && cg0 + tid < G4) {
      float4 s = red4[tid];
      for (int r = 1; r < RG; ++r) {
        const float4 t = red4[r * TPC + tid];
        s.x += t.x;
        s.y += t.y;
        s.z += t.z;
        s.w += t.w;
      }
      store_y4<T>(a.y, ri * CR + 4 * (cg0 + tid), s);
    }
    __syncthreads();
  }
  if (tid == 0) {
    const uint32_t old = atomicAdd(a.done, 1u);
    if (old == (uint32_t)a.n_red - 1) {
      atomicExch(a.arrive, 0u);
      atomicExch(a.done, 0u);
    }
  }
}

static int env_int(const char* name, int dflt) {
  const char* v = getenv(name);
  if (!v || !*v) return dflt;
  int x = atoi(v);
  return x > 0 ? x : dflt;
}

template <class T, int CPL, int P>
static hipError_t launch_mlp_kernel(const MlpArgs& a, size_t lds, hipStream_t stream) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)sparse_mlp_kernel<T, CPL, P>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((sparse_mlp_kernel<T, CPL, P>), dim3(a.n_wg), dim3(MLP_NT), lds, stream, a);
  return hipGetLastError();
}

template <class T, int P>
static hipError_t mlp_cpl(const MlpArgs& a, int cpl, size_t lds, hipStream_t stream) {
  if (cpl <= 1) return launch_mlp_kernel<T, 1, P>(a, lds, stream);
  if (cpl <= 2) return launch_mlp_kernel<T, 2, P>(a, lds, stream);
  if (cpl <= 4) return launch_mlp_kernel<T, 4, P>(a, lds, stream);
  return launch_mlp_kernel<T, 8, P>(a, lds, stream);
}

template <class T>
static hipError_t mlp_t(const np_shape& s, int layer, const void* x, const void* resident,
                        const int32_t* active_slots, int n_active, void* y, void* ws,
                        hipStream_t stream) {
  constexpr int V = T::V;
  MlpArgs a;
  a.NV = s.d_model / V;
  int P = 1;
  while (P < 4 && (a.NV + P - 1) / P > 512) P *= 2;
  a.NVP = (a.NV + P - 1) / P;
  const int cpl = (a.NVP + WAVE - 1) / WAVE;
  const int rpr = MLP_NW / P;
  const int max_wg = std::min(env_int("NP_MLP_MAX_WG", 256), MLP_MAX_WG);
  int n_wg = (n_active + rpr - 1) / rpr;
  if (n_wg > max_wg) n_wg = max_wg;
  if (n_wg < 1) n_wg = 1;
  a.rows_per_wg = n_active > 0 ? (n_active + n_wg - 1) / n_wg : 0;
  if (a.rows_per_wg > 0) n_wg = (n_active + a.rows_per_wg - 1) / a.rows_per_wg;
  a.n_wg = n_wg;
  int n_red = std::min(env_int("NP_MLP_NRED", 64), n_wg);
  int pw = 1;
  while (pw * 2 <= n_red) pw *= 2;
  n_red = pw;
  while (n_red > 1 && s.d_model % (4 * n_red) != 0) n_red /= 2;
  a.n_red = n_red;
  a.d = s.d_model;
  a.C = s.capacity;
  a.n_active = n_active;
  const size_t rec_vecs = (size_t)3 * a.NV;
  a.res_layer = (const uint4*)resident + (size_t)layer * s.capacity * rec_vecs;
  a.slots = active_slots;
  a.x = (const uint4*)x;
  a.y = y;
  a.partials = (float*)((char*)ws + ws_partials_offset(s));
  a.arrive = (uint32_t*)((char*)ws + WS_MLP_ARRIVE);
  a.done = (uint32_t*)((char*)ws + WS_MLP_DONE);
  a.ws = ws;
  size_t lds = (size_t)(MLP_NW / 2) * a.NVP * V * sizeof(float);
  if (lds < (size_t)MLP_NT * sizeof(float4)) lds = (size_t)MLP_NT * sizeof(float4);
  hipError_t e;
  switch (P) {
    case 1: e = mlp_cpl<T, 1>(a, cpl, lds, stream); break;
    case 2: e = mlp_cpl<T, 2>(a, cpl, lds, stream); break;
    default: e = mlp_cpl<T, 4>(a, cpl, lds, stream); break;
  }
  return e;
}

hipError_t launch_sparse_mlp(const np_shape& s, int layer, const void* x, const void* resident,
                             const int32_t* active_slots, int n_active, void* y, void* ws,
                             hipStream_t stream) {
  switch (s.wdtype) {
    case NP_F32: return mlp_t<TF32>(s, layer, x, resident, active_slots, n_active, y, ws, stream);
    case NP_F16: return mlp_t<TF16>(s, layer, x, resident, active_slots, n_active, y, ws, stream);
    default: return mlp_t<TBF16>(s, layer, x, resident, active_slots, n_active, y, ws, stream);
  }
}

}  // namespace np
