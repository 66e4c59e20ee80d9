// np_mlp.hip -- sparse gated MLP of one downstream layer over its resident
// active rows (Sec. 3.4: the slot map locates each active row, row order is
// irrelevant; Sec. 3.3: the down projection's output stays dense):
//     y = sum_j eq1(act(gate_j . x, up_j . x)) * downT_j
// with act ReLU-gated (max(g, 0) u) or SwiGLU (SiLU(g) u, Sec. 4) and eq1 the
// optional magnitude threshold of Sec. 3.2 (|a| < T -> 0).
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
// Reduction of the per-workgroup partials, one of two ways:
//  * single kernel (opt-in with NP_MLP_FUSED=1, when the whole grid fits on
//    the device at once; measured slower than two kernels at 7B shape):
//    the rows kernel writes its partial with agent-scope stores (coherent
//    across the XCDs' L2s without a cache write-back), meets every other
//    workgroup in a grid barrier (an arrival counter and a generation word in
//    the workspace; bounded spin, NP_DEVERR_SPIN_LIMIT when it runs out), and
//    then each workgroup reduces a slice of the columns over all partials
//    with agent-scope loads, in a fixed order, and rounds y once;
//  * two kernels (the default): the partials are stored in blocks of 16
//    columns and a separate reduce kernel sums each column's partials in
//    workgroup order; the kernel boundary makes them visible.
// Both orders are fixed, so each path is deterministic.
#include <stdlib.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <tuple>

#include "np_device.hpp"

namespace np {

struct MlpArgs {
  const uint4* res_layer;  // first record of the layer in the resident buffer
  const int32_t* slots;    // active_slots of the layer; nullptr: row j is slot j (dense layer)
  const uint4* x;
  float* partials;         // [d/16][n_wg][16] fp32
  void* ws;
  int n_active, C, NV, n_wg, P, PP, teams;  // PP: P rounded up to a power of two
  uint32_t layer_bytes;  // resident bytes of the layer (< 2^31)
  void* y;               // single-kernel path: the output
  const int32_t* n_dev;  // nullptr, or the row count at n_dev[layer] (<= n_active)
  int layer;
  int act;               // np_act
  const float* thr;      // nullptr, or the eq. 1 threshold of each layer at thr[layer]
  const int32_t* ids;    // with slots == nullptr: row j is slot slot_map[ids[j]]
  const int32_t* slot_map;
  int F;
};

// Slot of row r of the call: the active-slot list, the slot map of the
// active ids (an id outside [0, F) gives -1, reported as not resident), or
// the identity order of a dense layer.
__device__ inline int row_slot(const MlpArgs& a, int r, int b) {
  if (a.slots) return a.slots[r];
  if (a.ids) {
    const int id = a.ids[r];
    return (id >= 0 && id < a.F) ? a.slot_map[id] : -1;
  }
  return r * a.n_wg + b;
}


// Single-kernel path.  The partials use the blocked layout of the two-kernel
// path ([d/16][n_wg][16] fp32), written with agent-scope stores; after the
// grid barrier workgroup b reduces column blocks b, b + n_wg, ... with
// agent-scope loads, in the reduce kernel's order (thread t: 16-byte piece
// t % 4 of rows t/4, t/4 + nt/4, ...; a shuffle tree within each wave, then
// the waves in order).  The barrier's spin is bounded (polls of about 1 us
// each).
constexpr uint32_t MLP_SPIN_LIMIT = 1u << 20;

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

template <class T>
__device__ inline void store_y1(void* y, int col, float v) {
  if constexpr (T::dtype == NP_F32) ((float*)y)[col] = v;
  else ((uint16_t*)y)[col] = (uint16_t)T::from_f32(v);
}

// Grid barrier, then the column reduction of this workgroup's chunks.  Every
// thread of the workgroup calls it; thread 0 holds `gen0`, the generation
// read at entry.  red: blockDim.x float4 of LDS.
// Grid barrier over the n_wg workgroups of the launch: every thread calls
// it after its agent-scope stores; thread 0 holds `gen0`, the generation
// read at entry.  The last workgroup to arrive resets the arrival counter and
// advances the generation; the others poll it (bounded).
__device__ inline void grid_barrier(void* ws, int n_wg, int gen0) {
  __builtin_amdgcn_s_waitcnt(0);  // this wave's stores are complete
  __syncthreads();
  if (threadIdx.x == 0) {
    int* arrive = (int*)((char*)ws + WS_BAR_ARRIVE);
    int* gen = (int*)((char*)ws + WS_BAR_GEN);
    const int old = __hip_atomic_fetch_add(arrive, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old == n_wg - 1) {  // last to arrive: every workgroup's stores are done
      (void)__hip_atomic_exchange(arrive, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      (void)__hip_atomic_fetch_add(gen, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      uint32_t spins = 0;
      while (__hip_atomic_load(gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == gen0) {
        if (++spins == MLP_SPIN_LIMIT) {
          raise_error(ws, NP_DEVERR_SPIN_LIMIT);
          break;
        }
      }
    }
  }
  __syncthreads();
}

template <class T>
__device__ inline void fused_reduce(const MlpArgs& a, int gen0, float4* red) {
  grid_barrier(a.ws, a.n_wg, gen0);
  const int d = a.NV * T::V, nblk = (d + 15) / 16;
  const int t = threadIdx.x, nt = blockDim.x, lane = t & (WAVE - 1), w = t / WAVE;
  const int q = t & 3, rs = t >> 2, rstep = nt >> 2, nw = nt / WAVE;
  const __amdgpu_buffer_rsrc_t prs = make_rsrc(a.partials, (uint32_t)a.n_wg * nblk * 64u);
  for (int cb = blockIdx.x; cb < nblk; cb += a.n_wg) {
    const int col = cb * 16 + 4 * q;
    const bool cok = col < d;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int r0 = rs; r0 < a.n_wg; r0 += 4 * rstep) {  // rows in a fixed order
      float4 v[4];
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const int row = r0 + rstep * h;
        const uint32_t off = (row < a.n_wg && cok)
                                 ? (((uint32_t)cb * a.n_wg + row) * 16u + 4u * q) * 4u
                                 : BUF_OOB;
        v[h] = buf_load16_agent(prs, off);
      }
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        acc.x += v[h].x;
        acc.y += v[h].y;
        acc.z += v[h].z;
        acc.w += v[h].w;
      }
    }
#pragma unroll
    for (int m = 4; m < WAVE; m <<= 1) {
      acc.x += __shfl_xor(acc.x, m, WAVE);
      acc.y += __shfl_xor(acc.y, m, WAVE);
      acc.z += __shfl_xor(acc.z, m, WAVE);
      acc.w += __shfl_xor(acc.w, m, WAVE);
    }
    if (lane < 4) red[w * 4 + lane] = acc;
    __syncthreads();
    if (t < 4 && cok) {  // waves in order
      float4 o = red[t];
      for (int k = 1; k < nw; ++k) {
        o.x += red[k * 4 + t].x;
        o.y += red[k * 4 + t].y;
        o.z += red[k * 4 + t].z;
        o.w += red[k * 4 + t].w;
      }
      store_y4<T>(a.y, col, o);
    }
    __syncthreads();  // red is reused by the next block
  }
}

template <class T, int CPL, int R, int MAXT, bool FUSED>
__global__ __launch_bounds__(MAXT) void sparse_mlp_rows_kernel(MlpArgs a) {
  constexpr int V = T::V;
  // a round's R rows are finished in S stages of RS rows: the gate/up sums of
  // stage s are reduced, exchanged and applied while later stages' records
  // are still arriving (four stages for 8 rows over 9-10 waves, whose
  // exchange holds 2 * RS values of 16 lanes each in one wave)
  constexpr int S = (R >= 8 && MAXT > 512) ? 4 : (R >= 4 ? 2 : 1);
  constexpr int RS = R / S;
  constexpr int NVAL = 2 * RS;        // g and u of each stage row
  constexpr int G = WAVE / NVAL;      // lanes holding one reduced value
  __shared__ float gu[S][4][NVAL][16];  // stage, team, value, wave
  extern __shared__ float4 team_part[];  // (teams - 1) partial y of d floats
  const int lane = threadIdx.x & (WAVE - 1), wid = threadIdx.x / WAVE;
  const int P = a.P, teams = a.teams;
  const int team = wid / P, p = wid % P;
  const int b = blockIdx.x;
  int n_active = a.n_active;
  if (a.n_dev) {  // a row count produced on the device (variable-size sets)
    n_active = a.n_dev[a.layer];
    if (n_active < 0 || n_active > a.n_active) {
      if (threadIdx.x == 0 && b == 0) raise_error(a.ws, NP_DEVERR_STATE);
      n_active = n_active < 0 ? 0 : a.n_active;
    }
  }
  const float thr = a.thr ? a.thr[a.layer] : 0.f;  // eq. 1; 0 keeps every row
  // sparse: balanced contiguous ranges of the active list, workgroup b takes
  // [b*n/G, (b+1)*n/G).  Dense (no slot list): workgroup b takes rows b,
  // b + G, b + 2G, ... (index i of its range is row i*G + b), so the
  // workgroups of a round read neighbouring records together
  const bool dense = a.slots == nullptr && a.ids == nullptr;
  const int row_begin = dense ? 0 : (int)(((long long)b * n_active) / a.n_wg);
  const int row_end = dense ? n_active / a.n_wg + (b < n_active % a.n_wg ? 1 : 0)
                            : (int)(((long long)(b + 1) * n_active) / a.n_wg);
  const int v0 = p * WAVE * CPL;  // first vector of this wave's column slice
  int gen0 = 0;  // grid barrier generation at entry (thread 0)
  if (FUSED && threadIdx.x == 0)
    gen0 = __hip_atomic_load((int*)((char*)a.ws + WS_BAR_GEN), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);

  // first round's slots (lane r: row r) and x, both in flight before the
  // first wait
  int my_slot = -1;
  {
    const int r0 = row_begin + team * R;
    if (lane < R && r0 + lane < row_end) my_slot = row_slot(a, r0 + lane, b);
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
        gw[r][c] = buf_load16_nt(rsrc, off, 0);
        uw[r][c] = buf_load16_nt(rsrc, off, third);
        dw[r][c] = buf_load16_nt(rsrc, off, 2 * third);
      }
    }
    // next round's slots, in flight behind this round's records
    {
      const int rn = r0 + teams * R;
      my_slot = (lane < R && rn + lane < row_end) ? row_slot(a, rn + lane, b) : -1;
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
          float act = gated(a.act, gs[i], us[i]);
          if (fabsf(act) < thr) act = 0.f;
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
    if (team > 0) {
      if constexpr (!FUSED) return;
    } else {
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
  }
  // this wave's column slice of the workgroup's partial y (team 0)
  if (team == 0) {
    if constexpr (FUSED) {  // the blocked layout with agent-scope stores
      const uint32_t nblk = (uint32_t)(a.NV * V + 15) / 16u;
      const __amdgpu_buffer_rsrc_t prs = make_rsrc(a.partials, (uint32_t)a.n_wg * nblk * 64u);
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const uint32_t col0 = (uint32_t)(v0 + lane + WAVE * c) * V;
#pragma unroll
        for (int e = 0; e < V; e += 4) {
          const uint32_t col = col0 + e;
          const uint32_t off =
              vok[c] ? (((col >> 4) * (uint32_t)a.n_wg + b) * 16u + (col & 15u)) * 4u : BUF_OOB;
          buf_store16_agent(prs, off, make_float4(yacc[c][e], yacc[c][e + 1], yacc[c][e + 2],
                                                  yacc[c][e + 3]));
        }
      }
    } else {  // blocks of 16 columns: [d/16][n_wg][16] (see the reduce kernel),
              // nontemporal stores (measured 14.7 against 15.1 us per call)
      const uint32_t nblk = (uint32_t)(a.NV * V + 15) / 16u;
      const __amdgpu_buffer_rsrc_t prs = make_rsrc(a.partials, (uint32_t)a.n_wg * nblk * 64u);
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        const uint32_t col0 = (uint32_t)(v0 + lane + WAVE * c) * V;
#pragma unroll
        for (int e = 0; e < V; e += 4) {
          const uint32_t col = col0 + e;
          const uint32_t off =
              vok[c] ? (((col >> 4) * (uint32_t)a.n_wg + b) * 16u + (col & 15u)) * 4u : BUF_OOB;
          buf_store16_nt(prs, off, make_float4(yacc[c][e], yacc[c][e + 1], yacc[c][e + 2],
                                               yacc[c][e + 3]));
        }
      }
    }
  }
  if constexpr (FUSED) fused_reduce<T>(a, gen0, (float4*)team_part + (size_t)(teams - 1) * a.NV * V / 4);
}


// y[col] = sum over workgroups b of partial_b[col], in a fixed order.  The
// rows kernel stores the partials in blocks of 16 columns, [d/16][n_wg][16]
// fp32, so the block of 256 threads that owns 16 columns reads n_wg * 64
// contiguous bytes; the per-thread sums meet through a shuffle tree within
// each wave and then in wave order through LDS.
constexpr int RED_COLS = 16;

template <class T>
__global__ __launch_bounds__(256) void mlp_reduce_kernel(const float* __restrict__ partials,
                                                         int n_wg, int d, void* y) {
  // thread t reads 16-byte piece q = t % 4 of partial rows t / 4, t / 4 + 64,
  // ...: each wave instruction reads 1 KiB of contiguous memory
  __shared__ float4 red[4][4];  // wave, piece
  const int t = threadIdx.x, lane = t & (WAVE - 1), w = t / WAVE, q = t & 3, rs = t >> 2;
  const int col = blockIdx.x * RED_COLS + 4 * q;
  const bool cok = col < d;
  const float* blk = partials + (size_t)blockIdx.x * n_wg * RED_COLS + 4 * q;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int r0 = rs; r0 < n_wg; r0 += 256) {  // rows in a fixed order
    float4 v[4];
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const int row = r0 + 64 * h;
      v[h] = (row < n_wg && cok) ? *(const float4*)(blk + (size_t)row * RED_COLS)
                                 : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      acc.x += v[h].x;
      acc.y += v[h].y;
      acc.z += v[h].z;
      acc.w += v[h].w;
    }
  }
  // the wave's 16 row groups of each piece: a fixed shuffle tree over lane
  // bits 2..5, leaving lane q with piece q's wave sum
#pragma unroll
  for (int m = 4; m < WAVE; m <<= 1) {
    acc.x += __shfl_xor(acc.x, m, WAVE);
    acc.y += __shfl_xor(acc.y, m, WAVE);
    acc.z += __shfl_xor(acc.z, m, WAVE);
    acc.w += __shfl_xor(acc.w, m, WAVE);
  }
  if (lane < 4) red[w][lane] = acc;
  __syncthreads();
  if (t < 4 && cok) {  // waves in order
    float4 o = red[0][t];
#pragma unroll
    for (int k = 1; k < 4; ++k) {
      o.x += red[k][t].x;
      o.y += red[k][t].y;
      o.z += red[k][t].z;
      o.w += red[k][t].w;
    }
    store_y4<T>(y, col, o);
  }
}

// ---------------------------------------------------------------------------
// Single-kernel path without partial sums (16-bit records, whole wave
// slices).  Workgroup b owns (i) a balanced range of the active list, whose
// gate/up dot products it computes as the rows kernel does (wave p: a fixed
// 1 KiB column slice of gate and up; the sums meet in LDS) and turns into
// activations a_j, and (ii) a band of 16 columns of y.  At entry every thread
// also requests the band's 32 bytes of the down^T row of active rows t,
// t + nt, ..., so the down projection streams together with the gate/up
// rows instead of after them.  The activations are published with
// agent-scope stores; after a grid barrier each workgroup reads all of them
// and sums a_j * down_j[band] in a fixed order (thread, then wave): y needs no
// partial sums and no second kernel, and the result is deterministic.  Bands
// are handed out XCD by XCD (workgroups b, b + 8, ... run on one XCD and take
// adjacent bands), so the 128-byte lines of a down^T row are filled once per
// XCD, not once per band.  Needs the whole grid resident (checked at launch).
constexpr int CS_BAND = 16;  // columns of y per workgroup: two 16-byte vectors
constexpr int CS_RPT = 4;    // active rows per thread for the band (n <= 4 * threads)

template <class T, int R, int MAXT>
__global__ __launch_bounds__(MAXT) void sparse_mlp_colsplit_kernel(MlpArgs a) {
  constexpr int V = T::V;
  constexpr int BV = CS_BAND / V;   // vectors of a band row
  constexpr int NVAL = 2 * R;       // g and u of each row of a round
  constexpr int G = WAVE / NVAL;    // lanes holding one reduced value
  __shared__ float gu[NVAL][MAXT / WAVE];  // value, wave
  __shared__ float act_all[CS_RPT * MAXT];
  __shared__ float red[MAXT / WAVE][CS_BAND];
  const int lane = threadIdx.x & (WAVE - 1), p = threadIdx.x / WAVE;
  const int nt = blockDim.x, P = a.P, b = blockIdx.x;
  int n = a.n_active;
  if (a.n_dev) {  // a row count produced on the device (variable-size sets)
    n = a.n_dev[a.layer];
    if (n < 0 || n > a.n_active) {
      if (threadIdx.x == 0 && b == 0) raise_error(a.ws, NP_DEVERR_STATE);
      n = n < 0 ? 0 : a.n_active;
    }
  }
  const float thr = a.thr ? a.thr[a.layer] : 0.f;  // eq. 1; 0 keeps every row
  int gen0 = 0;
  if (threadIdx.x == 0)
    gen0 = __hip_atomic_load((int*)((char*)a.ws + WS_BAR_GEN), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
  const __amdgpu_buffer_rsrc_t rsrc = make_rsrc(a.res_layer, a.layer_bytes);
  const uint32_t third = (uint32_t)a.NV * 16u;
  // (ii) the band's piece of every active row's down^T, requested first
  const int band = (b % 8) * (a.n_wg / 8) + b / 8;
  const uint32_t band_off = 2u * third + (uint32_t)band * BV * 16u;
  int drow_slot[CS_RPT];
#pragma unroll
  for (int j = 0; j < CS_RPT; ++j) {
    const int row = threadIdx.x + nt * j;
    drow_slot[j] = row < n ? a.slots[row] : -1;
  }
  uint4 dv[CS_RPT][BV];
#pragma unroll
  for (int j = 0; j < CS_RPT; ++j) {
    const bool ok = drow_slot[j] >= 0 && drow_slot[j] < a.C;  // others reported by (i)
    const uint32_t base = ok ? (uint32_t)drow_slot[j] * 3u * third + band_off : BUF_OOB;
#pragma unroll
    for (int q = 0; q < BV; ++q) dv[j][q] = buf_load16_nt(rsrc, base, ok ? 16u * q : 0u);
  }
  // (i) the gate/up dot products of this workgroup's rows
  const int row_begin = (int)(((long long)b * n) / a.n_wg);
  const int row_end = (int)(((long long)(b + 1) * n) / a.n_wg);
  const int v = p * WAVE + lane;  // this lane's vector of the column slice
  const uint4 xr = a.x[v];
  const uint32_t loff = (uint32_t)v * 16u;
  float* avals = a.partials;  // the workspace's partial area holds the activations
  for (int rb = row_begin; rb < row_end; rb += R) {
    const int my_slot = (lane < R && rb + lane < row_end) ? a.slots[rb + lane] : -1;
    int slot[R];
    bool valid[R];
    bool bad = false;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      slot[r] = __builtin_amdgcn_readlane(my_slot, r);
      valid[r] = rb + r < row_end && slot[r] >= 0 && slot[r] < a.C;
      bad |= rb + r < row_end && !valid[r];
    }
    if (bad && threadIdx.x == 0) raise_error(a.ws, NP_DEVERR_NOT_RESIDENT);
    uint4 gw[R], uw[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const uint32_t roff = valid[r] ? (uint32_t)slot[r] * 3u * third + loff : BUF_OOB;
      gw[r] = buf_load16_nt(rsrc, roff, 0);
      uw[r] = buf_load16_nt(rsrc, roff, valid[r] ? third : 0u);
    }
    float val[NVAL];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      val[r] = T::dot(gw[r], xr, 0.f);
      val[R + r] = T::dot(uw[r], xr, 0.f);
    }
    wave_reduce_scatter<NVAL>(val);  // lane l holds the wave sum of value l / G
    if (lane % G == 0) gu[lane / G][p] = val[0];
    __syncthreads();
    if (threadIdx.x < R && rb + (int)threadIdx.x < row_end) {  // wave 0, lane r: row rb + r
      const int r = threadIdx.x;
      float g = 0.f, u = 0.f;
      for (int w = 0; w < P; ++w) {  // waves in order
        g += gu[r][w];
        u += gu[R + r][w];
      }
      const bool ok = my_slot >= 0 && my_slot < a.C;
      float act = ok ? gated(a.act, g, u) : 0.f;
      if (fabsf(act) < thr) act = 0.f;
      __hip_atomic_store((int*)(avals + rb + r), __float_as_int(act), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();  // gu is rewritten by the next round
  }
  grid_barrier(a.ws, a.n_wg, gen0);
  // every activation, from the agent-coherent level
  // whole 16-byte vectors (the area is larger; entries past n are not used)
  const __amdgpu_buffer_rsrc_t ars = make_rsrc(avals, (uint32_t)((n + 3) / 4) * 16u);
  for (int i = threadIdx.x; 4 * i < n; i += nt) {
    const float4 f = buf_load16_agent(ars, 16u * (uint32_t)i);
    act_all[4 * i] = f.x;
    act_all[4 * i + 1] = f.y;
    act_all[4 * i + 2] = f.z;
    act_all[4 * i + 3] = f.w;
  }
  __syncthreads();
  float acc[CS_BAND];
#pragma unroll
  for (int c = 0; c < CS_BAND; ++c) acc[c] = 0.f;
#pragma unroll
  for (int j = 0; j < CS_RPT; ++j) {
    const int row = threadIdx.x + nt * j;
    if (row < n && drow_slot[j] >= 0 && drow_slot[j] < a.C) {
      const float av = act_all[row];
#pragma unroll
      for (int q = 0; q < BV; ++q) T::axpy(acc + q * V, av, dv[j][q]);
    }
  }
  wave_reduce_scatter<CS_BAND>(acc);  // lane l: the wave's sum of column l / 4
  if (lane % (WAVE / CS_BAND) == 0) red[p][lane / (WAVE / CS_BAND)] = acc[0];
  __syncthreads();
  if (threadIdx.x < CS_BAND) {
    float y = 0.f;
    for (int w = 0; w < P; ++w) y += red[w][threadIdx.x];
    store_y1<T>(a.y, band * CS_BAND + threadIdx.x, y);
  }
}

static int env_int(const char* name, int dflt) {
  const char* v = getenv(name);
  if (!v || !*v) return dflt;
  int x = atoi(v);
  return x > 0 ? x : dflt;
}

// Workgroups of `kernel` that fit on the current device at once (cached).
static int coresident(const void* kernel, int threads, size_t lds) {
  static std::mutex mu;
  static std::map<std::tuple<int, const void*, int, size_t>, int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  std::lock_guard<std::mutex> g(mu);
  auto key = std::make_tuple(dev, kernel, threads, lds);
  auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, lds) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
    (void)hipGetLastError();
    per_cu = 0;
  }
  return cache[key] = per_cu * cus;
}

template <class T, int CPL, int R, int MAXT>
static void launch_rows_t(const MlpArgs& a, size_t lds, size_t lds_fused, bool want_fused,
                          bool* fused, hipStream_t stream) {
  const int threads = a.teams * a.P * WAVE;
  *fused = false;
  if (want_fused) {
    const void* k = (const void*)sparse_mlp_rows_kernel<T, CPL, R, MAXT, true>;
    if (a.n_wg <= coresident(k, threads, lds_fused)) {
      *fused = true;
      hipLaunchKernelGGL((sparse_mlp_rows_kernel<T, CPL, R, MAXT, true>), dim3(a.n_wg),
                         dim3(threads), lds_fused, stream, a);
      return;
    }
  }
  hipLaunchKernelGGL((sparse_mlp_rows_kernel<T, CPL, R, MAXT, false>), dim3(a.n_wg),
                     dim3(threads), lds, stream, a);
}

template <class T, int CPL, int R>
static void launch_rows(const MlpArgs& a, size_t lds, size_t lds_fused, bool want_fused,
                        bool* fused, hipStream_t stream) {
  const int threads = a.teams * a.P * WAVE;
  if (threads <= 512) {  // up to 8 waves: a register budget of 256 per lane
    launch_rows_t<T, CPL, R, 512>(a, lds, lds_fused, want_fused, fused, stream);
  } else if constexpr (R == 8) {  // 9-10 waves: 168 registers per lane
    if (threads <= 640) launch_rows_t<T, CPL, R, 640>(a, lds, lds_fused, want_fused, fused, stream);
  } else if constexpr (R <= 4) {  // 128 registers per lane: at most 4 rows a round
    launch_rows_t<T, CPL, R, 1024>(a, lds, lds_fused, want_fused, fused, stream);
  }
}

// Where one call keeps its scratch.  The workspace path: partials in dev_ws
// after the control block, opt-in single-kernel paths allowed.  The
// allocation-free path: partials in the library's own device array, at most
// max_wg workgroups, the error word the caller's, no opt-in path (they keep
// barrier words in the control block).
struct MlpScratch {
  float* partials;
  void* err;   // error word (raise_error target; WS_ERR is 0)
  int max_wg;
  bool opt_in;
};

template <class T>
static hipError_t mlp_t(const np_shape& s, int layer, const void* x, const void* resident,
                        const int32_t* active_slots, int n_active, void* y, void* ws,
                        hipStream_t stream, const int32_t* n_dev, const float* thr,
                        const MlpScratch* sc = nullptr, const int32_t* ids = nullptr,
                        const int32_t* slot_map = nullptr) {
  constexpr int V = T::V;
  MlpArgs a;
  a.ids = active_slots ? nullptr : ids;
  a.slot_map = slot_map;
  a.F = s.d_ffn;
  a.act = s.act;
  a.thr = thr;
  a.NV = s.d_model / V;
  // column slice per wave: 64 vectors (CPL = 1) while that needs at most 10
  // waves, else 128 vectors (CPL = 2; 70B, d 8192: 8 waves with 4-row rounds
  // take 33.6 us per call, 16 waves of 64 vectors 35.1)
  const int cpl = (a.NV + WAVE - 1) / WAVE <= 10 ? 1 : 2;
  a.P = (a.NV + WAVE * cpl - 1) / (WAVE * cpl);
  int teams = env_int("NP_MLP_TEAMS", 1);
  while (teams > 1 && teams * a.P > 16) teams /= 2;
  if (teams > 4) teams = 4;
  a.teams = teams;
  // rows per team and round: 8 while the workgroup has at most 10 waves
  // (168 or more registers per lane), 4 above that (128 registers), 2 for
  // 128-vector slices (13B, d 5120, 10 waves: 8-row rounds 19.14 us per
  // call, 4-row rounds 19.48)
  int R = cpl == 1 ? env_int("NP_MLP_R", teams * a.P <= 10 ? 8 : 4) : (teams * a.P <= 8 ? 4 : 2);
  // a small active set in 8-row rounds leaves most compute units idle: below
  // 128 such workgroups, 4-row rounds on twice as many stream faster (7B
  // shape, k = 550: 9.28 against 10.91 us per call; k = 1100, 138 workgroups
  // of 8 rows: 11.74 against 12.85 with 4-row rounds)
  if (R == 8 && !getenv("NP_MLP_R") && (n_active + 8 * teams - 1) / (8 * teams) < 128) R = 4;
  if (R != 2 && R != 4) R = 8;
  if (R == 8 && teams * a.P > 10) R = 4;
  a.PP = 1;
  while (a.PP < a.P) a.PP *= 2;
  // the exchange holds 2 * (R / stages) values x PP waves in one wave's lanes
  auto stage_rows = [&](int r) { return r >= 8 && teams * a.P > 8 ? r / 4 : (r >= 4 ? r / 2 : r); };
  while (R > 2 && 2 * stage_rows(R) * a.PP > WAVE) R /= 2;
  // at most one workgroup per CU (256), as many rounds of R rows per team
  // as 256 workgroups would need, and the fewest workgroups that still
  // finish in that many rounds: fewer, fuller workgroups finish sooner and
  // leave fewer partial sums (7B, k = 1651, one round: 207 workgroups take
  // 15.05 us per call, 256 take 15.45, and 206 or fewer, which need a second
  // round, about 18; 70B, k = 2867, three 4-row rounds: 239 workgroups 31.7
  // us, 256 32.0)
  const int per = R * teams;
  const int rounds = (n_active + per * 256 - 1) / (per * 256);
  const int full = rounds > 0 ? (n_active + per * rounds - 1) / (per * rounds) : 1;
  const int target = std::min(env_int("NP_MLP_WG", full), sc ? sc->max_wg : MLP_MAX_WG);
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
  a.partials = sc ? sc->partials : (float*)((char*)ws + ws_partials_offset(s));
  a.ws = sc ? sc->err : ws;
  a.y = y;
  a.n_dev = n_dev;
  a.layer = layer;
  // the single kernel without partial sums (opt-in, NP_MLP_COLSPLIT=1; measured
  // 17.3 against 16.1 us per call at the 7B shape: its 32-byte down^T pieces
  // touch 64 lines per load instruction and cost 4.5 us, the barrier 0.3 us)
  if constexpr (V == 8) {
    const bool on = (!sc || sc->opt_in) && env_int("NP_MLP_COLSPLIT", 0) == 1;
    const int P = a.NV / WAVE, bands = s.d_model / CS_BAND, threads = P * WAVE;
    if (on && active_slots && a.NV % WAVE == 0 && P <= 16 && bands % 8 == 0 &&
        n_active <= CS_RPT * threads && bands <= MLP_MAX_WG) {
      MlpArgs c = a;
      c.P = P;
      c.teams = 1;
      c.n_wg = bands;
      const void* k = threads <= 512 ? (const void*)sparse_mlp_colsplit_kernel<T, 8, 512>
                                     : (const void*)sparse_mlp_colsplit_kernel<T, 4, 1024>;
      if (bands <= coresident(k, threads, 0)) {
        if (threads <= 512)
          hipLaunchKernelGGL((sparse_mlp_colsplit_kernel<T, 8, 512>), dim3(bands), dim3(threads),
                             0, stream, c);
        else
          hipLaunchKernelGGL((sparse_mlp_colsplit_kernel<T, 4, 1024>), dim3(bands),
                             dim3(threads), 0, stream, c);
        return hipGetLastError();
      }
    }
  }
  const size_t lds = (size_t)(teams - 1) * a.NV * V * sizeof(float);
  // the single-kernel reduction adds one float4 per thread of LDS
  const size_t lds_fused = lds + (size_t)teams * a.P * WAVE * sizeof(float4);
  // single kernel on request, with at most 16 waves per workgroup (the
  // reduction's LDS); a co-resident grid is checked at launch
  const int threads = teams * a.P * WAVE;
  const bool want_fused =
      (!sc || sc->opt_in) && env_int("NP_MLP_FUSED", 0) == 1 && threads / WAVE <= 16;
  bool fused = false;
  if (cpl == 1) {
    if (R == 4) launch_rows<T, 1, 4>(a, lds, lds_fused, want_fused, &fused, stream);
    else if (R == 2) launch_rows<T, 1, 2>(a, lds, lds_fused, want_fused, &fused, stream);
    else launch_rows<T, 1, 8>(a, lds, lds_fused, want_fused, &fused, stream);
  } else {
    if (R == 4) launch_rows<T, 2, 4>(a, lds, lds_fused, want_fused, &fused, stream);
    else launch_rows<T, 2, 2>(a, lds, lds_fused, want_fused, &fused, stream);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || fused) return e;
  const int groups = (s.d_model + RED_COLS - 1) / RED_COLS;
  hipLaunchKernelGGL(mlp_reduce_kernel<T>, dim3(groups), dim3(256), 0, stream,
                     (const float*)a.partials, n_wg, s.d_model, y);
  return hipGetLastError();
}

// Dense layer (the dense prefix, Sec. 3.1): every one of the F records of
// `weights` ([F][3d]) is a row, in order; the rows kernel with the identity
// row -> record map.
hipError_t launch_dense_mlp(const np_shape& s, const void* weights, const void* x, void* y,
                            void* ws, hipStream_t stream) {
  np_shape d = s;
  d.capacity = s.d_ffn;  // the layer buffer is the whole layer
  return launch_sparse_mlp(d, 0, x, weights, nullptr, s.d_ffn, y, ws, stream);
}

hipError_t launch_sparse_mlp(const np_shape& s, int layer, const void* x, const void* resident,
                             const int32_t* active_slots, int n_active, void* y, void* ws,
                             hipStream_t stream, const int32_t* n_dev, const float* thr,
                             const int32_t* ids, const int32_t* slot_map) {
  switch (s.wdtype) {
    case NP_F32:
      return mlp_t<TF32>(s, layer, x, resident, active_slots, n_active, y, ws, stream, n_dev, thr,
                         nullptr, ids, slot_map);
    case NP_F16:
      return mlp_t<TF16>(s, layer, x, resident, active_slots, n_active, y, ws, stream, n_dev, thr,
                         nullptr, ids, slot_map);
    default:
      return mlp_t<TBF16>(s, layer, x, resident, active_slots, n_active, y, ws, stream, n_dev,
                          thr, nullptr, ids, slot_map);
  }
}

// ---------------------------------------------------------------------------
// Allocation-free sparse MLP (np_sparse_mlp_noalloc): the partial sums live in
// `scratch`, a file-scope device array of NOALLOC_SCRATCH_BYTES (room for
// NOALLOC_MAX_WG partial rows of NOALLOC_MAX_D fp32 columns), one copy per
// device, held until the process ends.  Host code never passes the array's
// name to a kernel: its device address is looked up once per device with
// hipGetSymbolAddress (with that device current) and kept in scratch_addr.
// Every call on a device shares that device's array; each call writes every
// partial row it reads before reading it, so nothing needs clearing, and two
// calls that overlap on one device race.
static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

static hipError_t scratch_addr(void** out) {
  static std::mutex mu;
  static void* addr[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

hipError_t launch_sparse_mlp_noalloc(const np_shape& s, int layer, const void* x,
                                     const void* resident, const int32_t* active_slots,
                                     int n_active, void* y, int32_t* dev_error,
                                     hipStream_t stream) {
  void* base = nullptr;
  hipError_t e = scratch_addr(&base);
  if (e != hipSuccess) return e;
  const MlpScratch sc{(float*)base, dev_error, NOALLOC_MAX_WG, false};
  switch (s.wdtype) {
    case NP_F32:
      return mlp_t<TF32>(s, layer, x, resident, active_slots, n_active, y, nullptr, stream,
                         nullptr, nullptr, &sc);
    case NP_F16:
      return mlp_t<TF16>(s, layer, x, resident, active_slots, n_active, y, nullptr, stream,
                         nullptr, nullptr, &sc);
    default:
      return mlp_t<TBF16>(s, layer, x, resident, active_slots, n_active, y, nullptr, stream,
                          nullptr, nullptr, &sc);
  }
}

}  // namespace np
