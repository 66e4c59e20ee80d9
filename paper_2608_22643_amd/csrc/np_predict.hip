// np_predict.hip -- low-rank activity predictor for all downstream layers
// (the one predictor pass after layer 0, Sec. 3.1 step 2 / Sec. 3.3):
//   z_l = A_l h        (r values per layer, fp32, kept in the workspace)
//   scores_l = B_l z_l (F values per layer, fp32)
// Both steps are batch-1 matrix-vector products: one weight element read per
// multiply-add, so they are bound by HBM bandwidth.  Weight rows are streamed
// with 16-byte loads that cover whole contiguous 1 KiB spans per wave
// instruction; there is no data reuse for matrix cores to exploit.
#include <stdlib.h>

#include "np_device.hpp"

namespace np {

// Stage 1: one wave per row of the stacked [L'*r][d] matrix A.  Lane i reads
// vectors i, i+64, ... of the row; UNROLL loads are issued before any math.
template <class T, int UNROLL>
__global__ __launch_bounds__(256) void predict_z_kernel(const uint4* __restrict__ A,
                                                        const uint4* __restrict__ h,
                                                        float* __restrict__ z, int rows,
                                                        int nv) {
  const int lane = threadIdx.x & (WAVE - 1);
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const uint4* a = A + (size_t)row * nv;
  float acc = 0.f;
  for (int base = lane; base < nv; base += WAVE * UNROLL) {
    uint4 wv[UNROLL], xv[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const int v = base + WAVE * u;
      if (v < nv) {
        wv[u] = load_nt(a + v);
        xv[u] = h[v];
      }
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      if (base + WAVE * u < nv) acc = T::dot(wv[u], xv[u], acc);
    }
  }
  acc = wave_sum(acc);
  if (lane == 0) z[row] = acc;
}

// Stage 2: scores[l][n] = B_l[n] . z_l.  A row of B is r elements (nvr
// 16-byte vectors).  A workgroup of 4 waves takes a block of SC_ROWS rows of
// one layer and stages z_l in LDS once.  Groups of 16 lanes own one row each
// (4 rows per wave instruction, 256 contiguous bytes per group); lane g of a
// group reads vectors g, g+16, ... (ZPL of them) and keeps the matching z
// values in registers.  Each wave walks its rows UNR row groups at a time,
// all loads of an iteration issued before any arithmetic.
// 64-row blocks: about 5,300 workgroups at 7B, so the last round of
// workgroups over the CUs is short (measured 6.5 TB/s against 6.0 with
// 256-row blocks).
constexpr int SC_ROWS = 64;

template <class T, int ZPL, int UNR>
__global__ __launch_bounds__(256) void predict_scores_kernel(const uint4* __restrict__ B,
                                                             const float* __restrict__ z,
                                                             float* __restrict__ scores,
                                                             int F, int r, int nvr) {
  constexpr int V = T::V;
  __shared__ float zs[16 * 8 * 8];  // r <= 128 vectors of 8 (or 4) elements
  const int lane = threadIdx.x & (WAVE - 1);
  const int wave = threadIdx.x >> 6;
  const int g = lane & 15, sub = lane >> 4;
  const int l = blockIdx.y;
  const float* zl = z + (size_t)l * r;
  for (int i = threadIdx.x; i < r; i += 256) zs[i] = zl[i];
  __syncthreads();
  float zr[ZPL][V];
#pragma unroll
  for (int i = 0; i < ZPL; ++i) {
    const int v = g + 16 * i;
#pragma unroll
    for (int e = 0; e < V; ++e) zr[i][e] = (v < nvr) ? zs[v * V + e] : 0.f;
  }
  const uint4* Bl = B + (size_t)l * F * nvr;
  float* sl = scores + (size_t)l * F;
  const int row_end = min(F, (int)(blockIdx.x + 1) * SC_ROWS);
  // wave w starts at row 4*UNR*w of the block; the 4 waves together advance 16*UNR rows
  for (int rb = blockIdx.x * SC_ROWS + wave * 4 * UNR; rb < row_end; rb += 16 * UNR) {
    uint4 wv[UNR][ZPL];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int n = rb + 4 * u + sub;
      const uint4* brow = Bl + (size_t)(n < row_end ? n : 0) * nvr;
#pragma unroll
      for (int i = 0; i < ZPL; ++i) {
        const int v = g + 16 * i;
        wv[u][i] = (n < row_end && v < nvr) ? load_nt(brow + v) : make_uint4(0u, 0u, 0u, 0u);
      }
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < ZPL; ++i) {
        float wf[V];
        T::unpack(wv[u][i], wf);
#pragma unroll
        for (int e = 0; e < V; ++e) acc = __builtin_fmaf(wf[e], zr[i][e], acc);
      }
      acc = group_sum<16>(acc);
      const int n = rb + 4 * u + sub;
      if (g == 0 && n < row_end) sl[n] = acc;
    }
  }
}

// ---------------------------------------------------------------------------
// The same two products on the matrix cores (selected with NP_PREDICT_MFMA=1,
// or by the caller's default, see launch_predict).  A batch-1 product uses
// one column of a 16 x 16 tile; the matrix unit replaces the per-lane dot
// products and the cross-lane sums (every row's sum comes out whole).
// ---------------------------------------------------------------------------

// z = A h: a workgroup of 4 waves owns a tile of 16 rows of the stacked
// [L'*r][d] matrix; wave w multiplies the tile over its quarter of the
// reduction steps (4V elements each; lane l loads 16 bytes of row l%16), h
// in column 0 of the B operand; the four waves' sums meet in LDS in wave
// order.  Out-of-range rows and elements are buffer loads with an
// out-of-range offset (zeros, no memory access).
template <class T, int UNR>
__global__ __launch_bounds__(256) void predict_z_mfma_kernel(const char* __restrict__ A,
                                                             const char* __restrict__ h,
                                                             float* __restrict__ z, int rows,
                                                             int d) {
  constexpr int V = T::V, KS = 4 * V, ES = 16 / V;
  __shared__ float part[4][16];
  const int lane = threadIdx.x & (WAVE - 1), w = threadIdx.x >> 6;
  const int row0 = blockIdx.x * 16, r = lane & 15, q = lane >> 4;
  const uint32_t row_bytes = (uint32_t)d * ES;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A + (size_t)row0 * row_bytes, 16u * row_bytes);
  const __amdgpu_buffer_rsrc_t rh = make_rsrc(h, row_bytes);
  const int steps = (d + KS - 1) / KS;
  const int s_begin = w * steps / 4, s_end = (w + 1) * steps / 4;
  const bool row_ok = row0 + r < rows;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = s_begin; s0 < s_end; s0 += UNR) {
    uint4 a[UNR], b[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int kk = (s0 + u) * KS + V * q;
      const bool ok = s0 + u < s_end && kk < d;
      a[u] = buf_load16_nt(ra, (ok && row_ok) ? (uint32_t)r * row_bytes + (uint32_t)kk * ES : BUF_OOB, 0);
      b[u] = buf_load16(rh, (ok && r == 0) ? (uint32_t)kk * ES : BUF_OOB, 0);
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) acc = mfma_step<T>(a[u], b[u], acc);
  }
  if (r == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) part[w][4 * q + i] = acc[i];
  }
  __syncthreads();
  if (threadIdx.x < 16 && row0 + (int)threadIdx.x < rows) {
    const int t = threadIdx.x;
    z[row0 + t] = ((part[0][t] + part[1][t]) + part[2][t]) + part[3][t];
  }
}

// scores_l = B_l z_l: a workgroup of 4 waves owns SC_ROWS rows of one layer,
// a 16-row tile per wave.  z is fp32 while the matrix unit takes 16-bit
// operands, so z_l is split into three 16-bit parts, z = hi + mid + lo
// (hi = z rounded, mid = the rest rounded, lo = what remains; 3 x 11 or
// 3 x 8 significand bits cover fp32's 24), placed in columns 0, 1, 2 of the
// B operand: the tile's products are exact in fp32 and the row's score is
// D[.][0] + D[.][1] + D[.][2].  For binary16 the layer's z is first scaled
// by 2^e (e from the largest |z|, so the parts stay in range; exact, undone
// on the result).  fp32 weights take z itself in column 0.
template <class T, int UNR>
__global__ __launch_bounds__(256) void predict_scores_mfma_kernel(const char* __restrict__ B,
                                                                  const float* __restrict__ z,
                                                                  float* __restrict__ scores,
                                                                  int F, int r) {
  constexpr int V = T::V, KS = 4 * V, ES = 16 / V;
  constexpr int NP = T::dtype == NP_F32 ? 1 : 3;
  constexpr int MAXK = 1024;  // r <= 1024 (16-bit) or 512 (fp32): whole steps
  __shared__ uint4 zp[NP][MAXK / V];
  __shared__ float wmax[4];
  const int lane = threadIdx.x & (WAVE - 1), w = threadIdx.x >> 6;
  const int rr = lane & 15, q = lane >> 4;
  const int l = blockIdx.y;
  const float* zl = z + (size_t)l * r;
  const int steps = (r + KS - 1) / KS;
  // the layer's scale (binary16 only)
  int e = 0;
  if constexpr (T::dtype == NP_F16) {
    float m = 0.f;
    for (int k = threadIdx.x; k < r; k += 256) m = fmaxf(m, fabsf(zl[k]));
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, WAVE));
    if (lane == 0) wmax[w] = m;
    __syncthreads();
    m = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
    if (m > 0.f && m <= 3.0e38f) e = 14 - ilogbf(m);
  }
  // the parts of z_l (zero past r), V elements per 16-byte vector
  for (int v = threadIdx.x; v < steps * 4; v += 256) {
    uint32_t pb[NP][V];
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const int k = v * V + j;
      float x = k < r ? ldexpf(zl[k], e) : 0.f;
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        pb[p][j] = T::from_f32(x);
        if constexpr (NP > 1) x -= T::lo(pb[p][j]);
      }
    }
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      if constexpr (V == 8)
        zp[p][v] = make_uint4(pb[p][0] | (pb[p][1] << 16), pb[p][2] | (pb[p][3] << 16),
                              pb[p][4] | (pb[p][5] << 16), pb[p][6] | (pb[p][7] << 16));
      else
        zp[p][v] = make_uint4(pb[p][0], pb[p][1], pb[p][2], pb[p][3]);
    }
  }
  __syncthreads();
  const int n0 = blockIdx.x * SC_ROWS + 16 * w;
  const uint32_t row_bytes = (uint32_t)r * ES;
  const __amdgpu_buffer_rsrc_t rb =
      make_rsrc(B + ((size_t)l * F + n0) * row_bytes, 16u * row_bytes);
  const bool row_ok = n0 + rr < F;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < steps; s0 += UNR) {
    uint4 a[UNR], b[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int kk = (s0 + u) * KS + V * q;
      const bool ok = s0 + u < steps;
      a[u] = buf_load16_nt(rb, (ok && row_ok && kk < r) ? (uint32_t)rr * row_bytes + (uint32_t)kk * ES
                                                       : BUF_OOB, 0);
      b[u] = (ok && rr < NP) ? zp[rr < NP ? rr : 0][(s0 + u) * 4 + q] : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) acc = mfma_step<T>(a[u], b[u], acc);
  }
  // column c of row i sits in lane 16 * (i / 4) + c: add columns 1 and 2
  // into column 0 (lo and mid first), undo the scale
  const float unscale = ldexpf(1.f, -e);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float v = acc[i];
    if constexpr (NP > 1) {
      const float c1 = __shfl_down(acc[i], 1, 16), c2 = __shfl_down(acc[i], 2, 16);
      v = (c2 + c1) + v;
    }
    const int n = n0 + 4 * q + i;
    if (rr == 0 && n < F) scores[(size_t)l * F + n] = v * unscale;
  }
}

// Row dot products out[i] = A[i] . x over rows of nv 16-byte vectors (the
// first stage of the predictor; also the centroid heads).
template <class T>
static hipError_t gemv_rows_t(const void* A, const void* x, float* out, int rows, int nv,
                              hipStream_t stream) {
  hipLaunchKernelGGL((predict_z_kernel<T, 8>), dim3((rows + 3) / 4), dim3(256), 0, stream,
                     (const uint4*)A, (const uint4*)x, out, rows, nv);
  return hipGetLastError();
}

hipError_t launch_centroid_logits(const np_shape& s, const np_centroid_model& m,
                                  const void* feat, float* logits, hipStream_t stream) {
  const int rows = 2 * s.layers * m.n_centroids;
  const int nv = m.feat_dim / vec_elems(s.wdtype);
  switch (s.wdtype) {
    case NP_F32: return gemv_rows_t<TF32>(m.heads, feat, logits, rows, nv, stream);
    case NP_F16: return gemv_rows_t<TF16>(m.heads, feat, logits, rows, nv, stream);
    default: return gemv_rows_t<TBF16>(m.heads, feat, logits, rows, nv, stream);
  }
}

static bool predict_mfma_requested() {
  const char* v = getenv("NP_PREDICT_MFMA");
  return v && atoi(v) == 1;
}

template <class T>
static hipError_t predict_mfma_t(const np_shape& s, const void* h, const void* A, const void* B,
                                 float* scores, void* ws, hipStream_t stream) {
  const int rows = s.layers * s.rank;
  float* z = (float*)((char*)ws + ws_z_offset());
  hipLaunchKernelGGL((predict_z_mfma_kernel<T, 8>), dim3((rows + 15) / 16), dim3(256), 0, stream,
                     (const char*)A, (const char*)h, z, rows, s.d_model);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 grid((s.d_ffn + SC_ROWS - 1) / SC_ROWS, s.layers);
  hipLaunchKernelGGL((predict_scores_mfma_kernel<T, 8>), grid, dim3(256), 0, stream,
                     (const char*)B, (const float*)z, scores, s.d_ffn, s.rank);
  return hipGetLastError();
}

template <class T>
static hipError_t predict_t(const np_shape& s, const void* h, const void* A, const void* B,
                            float* scores, void* ws, hipStream_t stream) {
  constexpr int V = T::V;
  if (predict_mfma_requested()) return predict_mfma_t<T>(s, h, A, B, scores, ws, stream);
  const int nv = s.d_model / V;
  const int rows = s.layers * s.rank;
  float* z = (float*)((char*)ws + ws_z_offset());
  hipLaunchKernelGGL((predict_z_kernel<T, 8>), dim3((rows + 3) / 4), dim3(256), 0, stream,
                     (const uint4*)A, (const uint4*)h, z, rows, nv);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nvr = s.rank / V;
  const int zpl = (nvr + 15) / 16;
  constexpr int UNR = 2;
  dim3 grid((s.d_ffn + SC_ROWS - 1) / SC_ROWS, s.layers);
#define NP_SCORES_CASE(Z)                                                                     \
  case Z:                                                                                     \
    hipLaunchKernelGGL((predict_scores_kernel<T, Z, UNR>), grid, dim3(256), 0, stream,        \
                       (const uint4*)B, (const float*)z, scores, s.d_ffn, s.rank, nvr);       \
    break;
  switch (zpl) {
    NP_SCORES_CASE(1)
    NP_SCORES_CASE(2)
    NP_SCORES_CASE(3)
    NP_SCORES_CASE(4)
    NP_SCORES_CASE(5)
    NP_SCORES_CASE(6)
    NP_SCORES_CASE(7)
    NP_SCORES_CASE(8)
    default:
      return hipErrorInvalidValue;  // rank beyond 128 vectors: rejected by validation
  }
#undef NP_SCORES_CASE
  return hipGetLastError();
}

hipError_t launch_predict(const np_shape& s, const void* h, const void* A, const void* B,
                          float* scores, void* ws, hipStream_t stream) {
  switch (s.wdtype) {
    case NP_F32: return predict_t<TF32>(s, h, A, B, scores, ws, stream);
    case NP_F16: return predict_t<TF16>(s, h, A, B, scores, ws, stream);
    default: return predict_t<TBF16>(s, h, A, B, scores, ws, stream);
  }
}

}  // namespace np
