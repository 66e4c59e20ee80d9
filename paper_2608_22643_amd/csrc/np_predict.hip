// np_predict.hip -- low-rank activity predictor for all downstream layers
// (the one predictor pass after layer 0, Sec. 3.1 step 2 / Sec. 3.3):
//   z_l = A_l h        (r values per layer, fp32, kept in the workspace)
//   scores_l = B_l z_l (F values per layer, fp32)
// Both steps are batch-1 matrix-vector products: one weight element read per
// multiply-add, so they are bound by HBM bandwidth.  Weight rows are streamed
// with 16-byte loads that cover whole contiguous 1 KiB spans per wave
// instruction; there is no data reuse for matrix cores to exploit.
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

template <class T>
static hipError_t predict_t(const np_shape& s, const void* h, const void* A, const void* B,
                            float* scores, void* ws, hipStream_t stream) {
  constexpr int V = T::V;
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
