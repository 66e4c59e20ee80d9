// np_mlp.hip -- sparse ReLU-gated MLP of one downstream layer over its
// resident active rows (Sec. 3.4: the slot map locates each active row, row
// order is irrelevant; Sec. 3.3: the down projection's output stays dense):
//     y = sum_j max(gate_j . x, 0) * (up_j . x) * downT_j
// Row j is one resident record [gate | up | downT] (3d contiguous elements),
// so the work is a stream of whole records: HBM-bound.
//
// Kernel 1 (rows): a workgroup owns a contiguous range of the active list.
// Its waves form `teams` row teams of P waves; each round, team j takes R
// rows of the range.  Within a team, wave p owns a fixed slice of the d
// columns (64*CPL 16-byte vectors of each of gate, up and downT), so
//   * every wave instruction reads 1 KiB of contiguous memory, and all
//     3*R*CPL loads of a round are issued before any arithmetic;
//   * the gate/up dot products of a row are P per-wave partial sums that
//     meet through a few bytes of LDS (fixed order);
//   * the wave's share of y (its column slice) stays in registers; the teams'
//     partial y meet once in LDS at the end (fixed order) and team 0 writes
//     the workgroup's partial y to the workspace.
// Kernel 2 (reduce): sums the per-workgroup partials of each column in
// workgroup order and rounds y once to the activation type.  The kernel
// boundary makes the partials visible across XCDs; no in-kernel fences.
#include <stdlib.h>

#include <algorithm>

#include "np_device.hpp"

namespace np {

struct MlpArgs {
  const uint4* res_layer;  // first record of the layer in the resident buffer
  const int32_t* slots;    // active_slots of the layer
  const uint4* x;
  float* partials;         // [n_wg][d]
  void* ws;
  int n_active, C, NV, n_wg, P, PP, teams;  // PP: P rounded up to a power of two
  uint32_t layer_bytes;  // resident bytes of the layer (< 2^31)
};

template <class T, int CPL, int R, int MAXT>
__global__ __launch_bounds__(MAXT) void sparse_mlp_rows_kernel(MlpArgs a) {
  constexpr int V = T::V;
  // a round's R rows are finished in S stages of RS rows: the gate/up sums of
  // stage s are reduced, exchanged and applied while later stages' records
  // are still arriving
  constexpr int S = R >= 4 ? 2 : 1;
  constexpr int RS = R / S;
  constexpr int NVAL = 2 * RS;        // g and u of each stage row
  constexpr int G = WAVE / NVAL;      // lanes holding one reduced value
  __shared__ float gu[S][4][NVAL][16];  // stage, team, value, wave
  extern __shared__ float4 team_part[];  // (teams - 1) partial y of d floats
  const int lane = threadIdx.x & (WAVE - 1), wid = threadIdx.x / WAVE;
  const int P = a.P, teams = a.teams;
  const int team = wid / P, p = wid % P;
  const int b = blockIdx.x;
  // balanced contiguous ranges: workgroup b takes rows [b*n/G, (b+1)*n/G)
  const int row_begin = (int)(((long long)b * a.n_active) / a.n_wg);
  const int row_end = (int)(((long long)(b + 1) * a.n_active) / a.n_wg);
  const int v0 = p * WAVE * CPL;  // first vector of this wave's column slice

  // first round's slots (lane r: row r) and x, both in flight before the
  // first wait
  int my_slot = -1;
  {
    const int r0 = row_begin + team * R;
    if (lane < R && r0 + lane < row_end) my_slot = a.slots[r0 + lane];
  }
  // Loads below are unconditional, with no branches around them, so the
  // compiler can wait for each stage's loads alone.  Record loads are buffer
  // loads: lanes past the slice and rows without a valid slot use an
  // out-of-range offset and read zeros without touching memory.
  const __amdgpu_buffer_rsrc_t rsrc = make_rsrc(a.res_layer, a.layer_bytes);
  const uint32_t third = (uint32_t)a.NV * 16u;
  uint4 xr[CPL];
  bool vok[CPL];
  uint32_t loff[CPL];  // this lane's byte offset within a third of a record
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int v = v0 + lane + WAVE * c;
    vok[c] = v < a.NV;
    loff[c] = vok[c] ? (uint32_t)v * 16u : BUF_OOB;
    xr[c] = a.x[vok[c] ? v : 0];
  }
  float yacc[CPL][V];
#pragma unroll
  for (int c = 0; c < CPL; ++c)
#pragma unroll
    for (int e = 0; e < V; ++e) yacc[c][e] = 0.f;

  // every wave runs the same number of rounds (barriers inside)
  for (int rb = row_begin; rb < row_end; rb += teams * R) {
    const int r0 = rb + team * R;
    int slot[R];
    bool valid[R];
    bool bad = false;  // a row of the active list without a resident slot
#pragma unroll
    for (int r = 0; r < R; ++r) {
      slot[r] = __builtin_amdgcn_readlane(my_slot, r);
      valid[r] = r0 + r < row_end && slot[r] >= 0 && slot[r] < a.C;
      bad |= r0 + r < row_end && !valid[r];
    }
    if (bad && threadIdx.x == 0) raise_error(a.ws, NP_DEVERR_NOT_RESIDENT);
    // all records of the round, in row order
    uint4 gw[R][CPL], uw[R][CPL], dw[R][CPL];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const uint32_t roff = valid[r] ? (uint32_t)slot[r] * 3u * third : BUF_OOB;
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const uint32_t off = roff + loff[c];  // both < 2^31: no wrap
        gw[r][c] = buf_load16(rsrc, off, 0);
        uw[r][c] = buf_load16(rsrc, off, third);
        dw[r][c] = buf_load16(rsrc, off, 2 * third);
      }
    }
    // next round's slots, in flight behind this round's records
    {
      const int rn = r0 + teams * R;
      my_slot = (lane < R && rn + lane < row_end) ? a.slots[rn + lane] : -1;
    }
#pragma unroll
    for (int st = 0; st < S; ++st) {
      float v[NVAL];
#pragma unroll
      for (int i = 0; i < RS; ++i) {
        const int r = st * RS + i;
        float g = 0.f, u = 0.f;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {  // lanes past the slice hold zeros
          g = T::dot(gw[r][c], xr[c], g);
          u = T::dot(uw[r][c], xr[c], u);
        }
        v[i] = g;
        v[RS + i] = u;
      }
      wave_reduce_scatter<NVAL>(v);  // lane l holds the wave sum of value l / G
      float gs[RS], us[RS];
      if (P > 1) {
        // the P waves' sums of each value meet in LDS; lane (value, wave)
        // reads one and a fixed shuffle tree over the PP lanes adds them
        if (lane % G == 0) gu[st][team][lane / G][p] = v[0];
        __syncthreads();
        const int PP = a.PP, val = lane / PP, q = lane % PP;
        float t = (val < NVAL && q < P) ? gu[st][team][val][q] : 0.f;
        for (int m = PP / 2; m >= 1; m >>= 1) t += __shfl_xor(t, m, WAVE);
#pragma unroll
        for (int i = 0; i < RS; ++i) {
          gs[i] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(t), i * PP));
          us[i] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(t), (RS + i) * PP));
        }
      } else {
#pragma unroll
        for (int i = 0; i < RS; ++i) {
          gs[i] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v[0]), i * G));
          us[i] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v[0]), (RS + i) * G));
        }
      }
#pragma unroll
      for (int i = 0; i < RS; ++i) {
        const int r = st * RS + i;
        if (valid[r]) {  // lanes past the slice accumulate values never written
          const float act = fmaxf(gs[i], 0.f) * us[i];
#pragma unroll
          for (int c = 0; c < CPL; ++c) T::axpy(yacc[c], act, dw[r][c]);
        }
      }
    }
    // with one stage, the next round's writes to gu must wait for this
    // round's reads (with two, the other stage's barrier orders them)
    if (S == 1 && P > 1) __syncthreads();
  }
  // teams 1.. hand their partial y to team 0 through LDS (fixed order)
  if (teams > 1) {
    if (team > 0) {
      float* dst = (float*)team_part + (size_t)(team - 1) * a.NV * V;
#pragma unroll
      for (int c = 0; c < CPL; ++c)
        if (vok[c]) {
          float4* d4 = (float4*)(dst + (size_t)(v0 + lane + WAVE * c) * V);
#pragma unroll
          for (int e = 0; e < V; e += 4)
            d4[e / 4] = make_float4(yacc[c][e], yacc[c][e + 1], yacc[c][e + 2], yacc[c][e + 3]);
        }
    }
    __syncthreads();
    if (team > 0) return;
    for (int t = 1; t < teams; ++t) {
      const float* src = (const float*)team_part + (size_t)(t - 1) * a.NV * V;
#pragma unroll
      for (int c = 0; c < CPL; ++c)
        if (vok[c]) {
          const float4* s4 = (const float4*)(src + (size_t)(v0 + lane + WAVE * c) * V);
#pragma unroll
          for (int e = 0; e < V; e += 4) {
            const float4 q = s4[e / 4];
            yacc[c][e] += q.x;
            yacc[c][e + 1] += q.y;
            yacc[c][e + 2] += q.z;
            yacc[c][e + 3] += q.w;
          }
        }
    }
  }
  // this wave's column slice of the workgroup's partial y
  float* dst = a.partials + (size_t)b * a.NV * V;
#pragma unroll
  for (int c = 0; c < CPL; ++c)
    if (vok[c]) {
      float4* d4 = (float4*)(dst + (size_t)(v0 + lane + WAVE * c) * V);
#pragma unroll
      for (int e = 0; e < V; e += 4)
        d4[e / 4] = make_float4(yacc[c][e], yacc[c][e + 1], yacc[c][e + 2], yacc[c][e + 3]);
    }
}

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

// y[col] = sum over workgroups b of partials[b][col], in a fixed order.  A
// block of 256 threads owns 16 columns; thread t loads 64 contiguous bytes
// of each of the partial rows t, t+256, t+512, t+768 (all loads in flight at
// once).  Each wave then reduce-scatters its 16 column sums, and one lane per
// column adds the four waves' sums in wave order.
constexpr int RED_COLS = 16;

template <class T>
__global__ __launch_bounds__(256) void mlp_reduce_kernel(const float* __restrict__ partials,
                                                         int n_wg, int d, void* y) {
  __shared__ float red[4][RED_COLS];
  const int t = threadIdx.x, lane = t & (WAVE - 1), w = t / WAVE;
  const int col = blockIdx.x * RED_COLS;
  float4 v[4][RED_COLS / 4];
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const int row = t + 256 * h;
#pragma unroll
    for (int q = 0; q < RED_COLS / 4; ++q)
      v[h][q] = (row < n_wg && col + 4 * q < d)
                    ? *(const float4*)(partials + (size_t)row * d + col + 4 * q)
                    : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float s[RED_COLS];
#pragma unroll
  for (int q = 0; q < RED_COLS / 4; ++q) {
    float4 a = v[0][q];
#pragma unroll
    for (int h = 1; h < 4; ++h) {
      a.x += v[h][q].x;
      a.y += v[h][q].y;
      a.z += v[h][q].z;
      a.w += v[h][q].w;
    }
    s[4 * q] = a.x;
    s[4 * q + 1] = a.y;
    s[4 * q + 2] = a.z;
    s[4 * q + 3] = a.w;
  }
  wave_reduce_scatter<RED_COLS>(s);  // lane l: wave sum of column l / 4
  if (lane % (WAVE / RED_COLS) == 0) red[w][lane / (WAVE / RED_COLS)] = s[0];
  __syncthreads();
  if (t < RED_COLS / 4 && col + 4 * t < d) {
    float4 o;
    float* of = (float*)&o;
#pragma unroll
    for (int j = 0; j < 4; ++j) of[j] = red[0][4 * t + j] + red[1][4 * t + j] + red[2][4 * t + j] + red[3][4 * t + j];
    store_y4<T>(y, col + 4 * t, o);
  }
}

static int env_int(const char* name, int dflt) {
  const char* v = getenv(name);
  if (!v || !*v) return dflt;
  int x = atoi(v);
  return x > 0 ? x : dflt;
}

template <class T, int CPL, int R>
static void launch_rows(const MlpArgs& a, int n_wg, size_t lds, hipStream_t stream) {
  const int threads = a.teams * a.P * WAVE;
  if (threads <= 512) {  // up to 8 waves: a register budget of 256 per lane
    hipLaunchKernelGGL((sparse_mlp_rows_kernel<T, CPL, R, 512>), dim3(n_wg), dim3(threads), lds,
                       stream, a);
  } else if constexpr (R <= 4) {  // 128 registers per lane: at most 4 rows a round
    hipLaunchKernelGGL((sparse_mlp_rows_kernel<T, CPL, R, 1024>), dim3(n_wg), dim3(threads), lds,
                       stream, a);
  }
}

template <class T>
static hipError_t mlp_t(const np_shape& s, int layer, const void* x, const void* resident,
                        const int32_t* active_slots, int n_active, void* y, void* ws,
                        hipStream_t stream) {
  constexpr int V = T::V;
  MlpArgs a;
  a.NV = s.d_model / V;
  // column slice per wave: 64 vectors (CPL = 1) while that needs at most 16
  // waves, else 128 vectors (CPL = 2)
  const int cpl = (a.NV + WAVE - 1) / WAVE <= 16 ? 1 : 2;
  a.P = (a.NV + WAVE * cpl - 1) / (WAVE * cpl);
  int teams = env_int("NP_MLP_TEAMS", 1);
  while (teams > 1 && teams * a.P > 16) teams /= 2;
  if (teams > 4) teams = 4;
  a.teams = teams;
  // rows per team and round: 8 while the workgroup has at most 8 waves (256
  // registers per lane), 4 above that (128 registers), 2 for 128-vector slices
  int R = cpl == 1 ? env_int("NP_MLP_R", teams * a.P <= 8 ? 8 : 4) : 2;
  if (R != 2 && R != 4) R = 8;
  if (R == 8 && teams * a.P > 8) R = 4;
  a.PP = 1;
  while (a.PP < a.P) a.PP *= 2;
  // the exchange holds 2 * (R / stages) values x PP waves in one wave's lanes
  while (R > 2 && 2 * (R >= 4 ? R / 2 : R) * a.PP > WAVE) R /= 2;
  // one workgroup per CU by default: the bytes of each CU, not the total,
  // set the time of this short streaming kernel, so spread rows evenly
  const int target = std::min(env_int("NP_MLP_WG", 256), MLP_MAX_WG);
  int n_wg = n_active < target ? n_active : target;
  if (n_wg < 1) n_wg = 1;
  a.n_wg = n_wg;
  a.n_active = n_active;
  a.C = s.capacity;
  const size_t rec_vecs = (size_t)3 * a.NV;
  a.res_layer = (const uint4*)resident + (size_t)layer * s.capacity * rec_vecs;
  a.layer_bytes = (uint32_t)((size_t)s.capacity * rec_vecs * 16);
  a.slots = active_slots;
  a.x = (const uint4*)x;
  a.partials = (float*)((char*)ws + ws_partials_offset(s));
  a.ws = ws;
  const size_t lds = (size_t)(teams - 1) * a.NV * V * sizeof(float);
  if (cpl == 1) {
    if (R == 4) launch_rows<T, 1, 4>(a, n_wg, lds, stream);
    else if (R == 2) launch_rows<T, 1, 2>(a, n_wg, lds, stream);
    else launch_rows<T, 1, 8>(a, n_wg, lds, stream);
  } else {
    launch_rows<T, 2, 2>(a, n_wg, lds, stream);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int groups = (s.d_model + RED_COLS - 1) / RED_COLS;
  hipLaunchKernelGGL(mlp_reduce_kernel<T>, dim3(groups), dim3(256), 0, stream,
                     (const float*)a.partials, n_wg, s.d_model, y);
  return hipGetLastError();
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
