// np_calib.hip -- the magnitude-threshold sparsity of Sec. 3.2 (eq. 1):
//  * act_batch_kernel: activations A(i, l) = act(G x_i, U x_i) of one layer
//    over a batch of calibration tokens, on the matrix cores;
//  * pct_hist_kernel / pct_select_kernel (percentile_kernel for short rows):
//    per layer, the nearest-rank alpha-th percentile of |A| (the threshold
//    T(l, alpha)) by radix selection;
//  * threshold_active_kernel: eq. 1 as an active set, |a| >= T, in the
//    selection's mask + ascending-id layout.
#include "np_device.hpp"

namespace np {

// ---------------------------------------------------------------------------
// activations of a token batch
// ---------------------------------------------------------------------------
// The gate and up projections of a batch are two matrix products, G X^T and
// U X^T (neurons x tokens, reduction over d), so they run on MFMA with fp32
// accumulation: 16 x 16 output tiles, each a v_mfma_f32_16x16x32 (16-bit
// types) or four v_mfma_f32_16x16x4f32 (fp32) per "step" of 4*V reduction
// elements.  Lane l holds row l%16 of the A operand (a neuron's gate or up
// row) and column l%16 of the B operand (a token), each as the V consecutive
// elements starting at step*4V + V*(l/16), so the two operands pair the same
// reduction indices whatever order the unit sums them in, and one 16-byte
// load instruction reads 64 contiguous bytes of each of 16 rows.  The
// accumulator layout: lane l, register r holds output row 4*(l/16) + r
// (neuron) and column l%16 (token).
//
// A workgroup owns 64 neurons (four row tiles) and every token of the launch
// (up to 128: eight 16-token tiles); wave w takes token tiles w and w + 4 of
// every row tile over the whole reduction, so no wave needs another's sums,
// and each token fragment a wave loads serves four row tiles.  The neurons' gate and up
// rows, and the chunk's token rows, stream through LDS in chunks of KC
// elements: the workgroup loads a chunk with whole-line 16-byte loads (16
// lanes per 256-byte row piece) into one of two buffers while the waves
// multiply the other, and each wave reads its MFMA fragments from LDS (rows
// padded by 16 bytes: no bank conflicts).
constexpr int AB_WAVES = 4;
constexpr int AB_NB = 64;         // neurons of a workgroup (AB_NB / 16 row tiles)
constexpr int AB_MAX_TILES = 8;   // token tiles of 16
constexpr int AB_ROWB = 256;      // bytes of a row piece per chunk
constexpr int AB_PITCH = AB_ROWB + 16;

struct ActBatchArgs {
  const void* w;    // one layer's [F][3d] records
  const void* x;    // [n][d] tokens of this launch
  float* acts;      // [n][F] rows of this launch
  uint32_t w_bytes, x_bytes;
  int F, d, n, act;
};

template <class T, int TPW>
__global__ __launch_bounds__(AB_WAVES * WAVE) void act_batch_kernel(ActBatchArgs a) {
  constexpr int V = T::V, ESZ = 16 / V, KS = 4 * V;  // KS: reduction elements per MFMA step
  constexpr int KC = AB_ROWB / ESZ;                  // reduction elements per chunk
  constexpr int SPC = KC / KS;                       // MFMA steps per chunk (4)
  constexpr int MT = AB_NB / 16;                      // row tiles
  constexpr int PIECES = 2 * AB_NB * (AB_ROWB / 16);  // 16-byte pieces of a chunk (g and u)
  constexpr int PPT = PIECES / (AB_WAVES * WAVE);    // pieces per thread (8)
  __shared__ __attribute__((aligned(16))) char lds[2][2][AB_NB][AB_PITCH];  // buffer, g/u, row
  // the chunk's token pieces: buffer, token, 16-byte column (padded rows)
  __shared__ __attribute__((aligned(16))) char xs[2][16 * AB_MAX_TILES][AB_PITCH];
  constexpr int XPT = 16 * AB_MAX_TILES * (AB_ROWB / 16) / (AB_WAVES * WAVE);  // token pieces per thread (8)
  const int t = threadIdx.x, lane = t & (WAVE - 1), w = t / WAVE, grp = lane / 16;
  const int n0 = blockIdx.x * AB_NB;
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.w, a.w_bytes), xr = make_rsrc(a.x, a.x_bytes);
  const uint32_t rec = (uint32_t)(3 * a.d * ESZ), dbytes = (uint32_t)(a.d * ESZ);
  const int chunks = (a.d + KC - 1) / KC;
  // this thread's pieces of every chunk: piece p -> (projection, row, 16-byte column)
  uint32_t p_off[PPT];  // byte offset at reduction index 0, or OOB
  int p_col[PPT];
#pragma unroll
  for (int i = 0; i < PPT; ++i) {
    const int pc = t + AB_WAVES * WAVE * i;
    const int proj = pc / (PIECES / 2), row = (pc / (AB_ROWB / 16)) % AB_NB, col = pc % (AB_ROWB / 16);
    const int neuron = n0 + row;
    p_off[i] = neuron < a.F ? (uint32_t)neuron * rec + (uint32_t)proj * dbytes : BUF_OOB;
    p_col[i] = col;
  }
  auto load_chunk = [&](int c, uint4* r) {
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int k = c * KC + p_col[i] * V;  // first element of the piece
      r[i] = buf_load16_nt(wr, (p_off[i] != BUF_OOB && k < a.d) ? p_off[i] + (uint32_t)k * ESZ
                                                             : BUF_OOB, 0);
    }
  };
  auto store_chunk = [&](int buf, const uint4* r) {
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int pc = t + AB_WAVES * WAVE * i;
      const int proj = pc / (PIECES / 2), row = (pc / (AB_ROWB / 16)) % AB_NB, col = pc % (AB_ROWB / 16);
      *(uint4*)&lds[buf][proj][row][col * 16] = r[i];
    }
  };
  // the chunk's token pieces, whole 256-byte row pieces per 16 lanes like
  // the weights (a fragment load straight from memory would touch 16 token
  // rows per instruction): piece p -> token p / 16, 16-byte column p % 16
  uint32_t x_off[XPT];  // byte offset at reduction index 0, or OOB
#pragma unroll
  for (int i = 0; i < XPT; ++i) {
    const int pc = t + AB_WAVES * WAVE * i, tok = pc / (AB_ROWB / 16);
    x_off[i] = tok < a.n ? (uint32_t)tok * dbytes : BUF_OOB;
  }
  auto load_xchunk = [&](int c, uint4* r) {
#pragma unroll
    for (int i = 0; i < XPT; ++i) {
      const int pc = t + AB_WAVES * WAVE * i;
      const int k = c * KC + (pc % (AB_ROWB / 16)) * V;
      r[i] = buf_load16(xr, (x_off[i] != BUF_OOB && k < a.d) ? x_off[i] + (uint32_t)k * ESZ
                                                             : BUF_OOB, 0);
    }
  };
  auto store_xchunk = [&](int buf, const uint4* r) {
#pragma unroll
    for (int i = 0; i < XPT; ++i) {
      const int pc = t + AB_WAVES * WAVE * i;
      *(uint4*)&xs[buf][pc / (AB_ROWB / 16)][(pc % (AB_ROWB / 16)) * 16] = r[i];
    }
  };
  f32x4 accg[MT][TPW], accu[MT][TPW];
#pragma unroll
  for (int m = 0; m < MT; ++m)
#pragma unroll
    for (int j = 0; j < TPW; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) accg[m][j][r] = accu[m][j][r] = 0.f;

  uint4 pre[PPT], prex[XPT];
  load_chunk(0, pre);
  load_xchunk(0, prex);
  store_chunk(0, pre);
  store_xchunk(0, prex);
  __syncthreads();
  for (int c = 0; c < chunks; ++c) {
    const int buf = c & 1;
    if (c + 1 < chunks) {  // the next chunk is in flight during this one's products
      load_chunk(c + 1, pre);
      load_xchunk(c + 1, prex);
    }
#pragma unroll
    for (int s = 0; s < SPC; ++s) {
      uint4 b[TPW];  // token tile w + 4j: token 16 (w + 4j) + lane % 16
#pragma unroll
      for (int j = 0; j < TPW; ++j)
        b[j] = *(const uint4*)&xs[buf][(w + AB_WAVES * j) * 16 + (lane & 15)][s * 64 + grp * 16];
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const int row = 16 * m + (lane & 15);
        const uint4 ag = *(const uint4*)&lds[buf][0][row][s * 64 + grp * 16];
        const uint4 au = *(const uint4*)&lds[buf][1][row][s * 64 + grp * 16];
#pragma unroll
        for (int j = 0; j < TPW; ++j) {
          accg[m][j] = mfma_step<T>(ag, b[j], accg[m][j]);
          accu[m][j] = mfma_step<T>(au, b[j], accu[m][j]);
        }
      }
    }
    if (c + 1 < chunks) {
      store_chunk(buf ^ 1, pre);
      store_xchunk(buf ^ 1, prex);
    }
    __syncthreads();  // the other buffer is complete; this one may be overwritten next
  }
  // acts[token][neuron]: lane l, register r holds neuron 16 m + 4 (l / 16) + r
#pragma unroll
  for (int j = 0; j < TPW; ++j) {
    const int tok = (w + AB_WAVES * j) * 16 + (lane & 15);
    if (tok >= a.n) continue;
    float* dst = a.acts + (size_t)tok * a.F;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const int nb = n0 + 16 * m + 4 * grp;  // neurons nb .. nb + 3
      float o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = gated(a.act, accg[m][j][e], accu[m][j][e]);
      if ((a.F & 3) == 0) {
        if (nb < a.F) *(float4*)(dst + nb) = make_float4(o[0], o[1], o[2], o[3]);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (nb + e < a.F) dst[nb + e] = o[e];
      }
    }
  }
}

template <class T>
static hipError_t act_batch_t(const np_shape& s, const void* weights, const void* x, int n,
                              float* acts, hipStream_t stream) {
  constexpr int ESZ = 16 / T::V;
  const int tiles = (s.d_ffn + AB_NB - 1) / AB_NB;
  for (int i0 = 0; i0 < n; i0 += 16 * AB_MAX_TILES) {
    ActBatchArgs a;
    a.w = weights;
    a.x = (const char*)x + (size_t)i0 * s.d_model * ESZ;
    a.acts = acts + (size_t)i0 * s.d_ffn;
    a.n = std::min(n - i0, 16 * AB_MAX_TILES);
    a.w_bytes = (uint32_t)((size_t)s.d_ffn * 3 * s.d_model * ESZ);
    a.x_bytes = (uint32_t)((size_t)a.n * s.d_model * ESZ);
    a.F = s.d_ffn;
    a.d = s.d_model;
    a.act = s.act;
    const int ntt = (a.n + 15) / 16;  // token tiles; wave w takes tiles w, w + 4
    if (ntt <= AB_WAVES)
      hipLaunchKernelGGL((act_batch_kernel<T, 1>), dim3(tiles), dim3(AB_WAVES * WAVE), 0, stream,
                         a);
    else
      hipLaunchKernelGGL((act_batch_kernel<T, 2>), dim3(tiles), dim3(AB_WAVES * WAVE), 0, stream,
                         a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_act_batch(const np_shape& s, const void* weights, const void* x, int n,
                            float* acts, hipStream_t stream) {
  switch (s.wdtype) {
    case NP_F32: return act_batch_t<TF32>(s, weights, x, n, acts, stream);
    case NP_F16: return act_batch_t<TF16>(s, weights, x, n, acts, stream);
    default: return act_batch_t<TBF16>(s, weights, x, n, acts, stream);
  }
}

// ---------------------------------------------------------------------------
// per-row nearest-rank percentile of the magnitudes
// ---------------------------------------------------------------------------
// The magnitude's bits (sign cleared) order non-negative floats like
// integers, so the m-th smallest magnitude is found digit by digit from the
// top: 11, 10 and 10 bits.  Each pass streams the row once, counts the
// values that match the digits decided so far into a histogram of the next
// digit (four LDS copies, by wave, against atomic contention on the few bins
// a narrow exponent range fills), and a prefix sum over the bins finds the
// digit that holds the m-th value.
constexpr int PCT_NT = 1024;
constexpr int PCT_BINS = 2048;
constexpr int PCT_COPIES = 4;

template <bool V4>
__global__ __launch_bounds__(PCT_NT) void percentile_kernel(const float* __restrict__ values,
                                                            int64_t n, int64_t m, float* out,
                                                            void* ws) {
  __shared__ uint32_t hist[PCT_COPIES][PCT_BINS];
  __shared__ uint32_t scan[PCT_NT / WAVE + 1];
  __shared__ uint32_t sel[2];  // chosen digit, rank left within it
  const int tid = threadIdx.x, copy = (tid / WAVE) % PCT_COPIES;
  const float* row = values + (size_t)blockIdx.x * (size_t)n;
  uint32_t prefix = 0, known = 0;  // decided high bits and their mask
  uint32_t rank = (uint32_t)m;     // 1-based rank within the matching values
  bool nan = false;
  const int shifts[3] = {20, 10, 0}, widths[3] = {11, 10, 10};
  for (int pass = 0; pass < 3; ++pass) {
    const int sh = shifts[pass], nb = 1 << widths[pass];
    for (int i = tid; i < PCT_COPIES * PCT_BINS; i += PCT_NT) (&hist[0][0])[i] = 0u;
    __syncthreads();
    auto count = [&](float v) {
      const uint32_t key = __float_as_uint(v) & 0x7FFFFFFFu;
      if (pass == 0 && key > 0x7F800000u) nan = true;
      if ((key & known) == prefix) atomicAdd(&hist[copy][(key >> sh) & (nb - 1)], 1u);
    };
    if constexpr (V4) {
      const float4* r4 = (const float4*)row;
      for (int64_t i = tid; i < n / 4; i += PCT_NT) {
        const float4 v = r4[i];
        count(v.x);
        count(v.y);
        count(v.z);
        count(v.w);
      }
    } else {
      for (int64_t i = tid; i < n; i += PCT_NT) count(row[i]);
    }
    __syncthreads();
    // thread t owns bins 2t, 2t + 1
    uint32_t c[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int b = 2 * tid + j;
      c[j] = 0u;
      if (b < nb)
#pragma unroll
        for (int cp = 0; cp < PCT_COPIES; ++cp) c[j] += hist[cp][b];
    }
    uint32_t tot;
    const uint32_t before = block_excl_scan<PCT_NT>(c[0] + c[1], scan, &tot);
    if (before < rank && rank <= before + c[0]) {
      sel[0] = 2 * tid;
      sel[1] = rank - before;
    } else if (before + c[0] < rank && rank <= before + c[0] + c[1]) {
      sel[0] = 2 * tid + 1;
      sel[1] = rank - before - c[0];
    }
    __syncthreads();
    prefix |= sel[0] << sh;
    known |= (uint32_t)(nb - 1) << sh;
    rank = sel[1];
    __syncthreads();  // sel and hist are rewritten by the next pass
  }
  if (nan) raise_error(ws, NP_DEVERR_NAN_SCORE);
  if (tid == 0) out[blockIdx.x] = __uint_as_float(prefix);
}

// The same selection spread over many workgroups per row, for long rows:
// each pass is a histogram kernel over (slice, row) workgroups, which count
// their slice of the row into LDS and add the nonzero bins to the row's
// histogram in dev_ws, and a selection kernel with one workgroup per row,
// which scans that histogram, narrows the row's (prefix, known bits, rank)
// state and clears the histogram for the next pass.  The kernel boundaries
// order the passes.  dev_ws layout past the control block: state [rows][4]
// uint32, then histograms [rows][PCT_BINS] uint32.
constexpr int PCT_HNT = 512;
constexpr int PCT_HCOPIES = 4;  // LDS histogram copies, by wave

__host__ __device__ inline size_t pct_hist_offset(int rows) {
  return (WS_CTRL_BYTES + (size_t)rows * 16 + 255) & ~(size_t)255;
}
size_t percentile_ws_bytes(int rows) {
  return pct_hist_offset(rows) + (size_t)rows * PCT_BINS * 4;
}

__global__ __launch_bounds__(256) void pct_init_kernel(int64_t m, void* ws) {
  const int row = blockIdx.x;
  uint32_t* st = (uint32_t*)((char*)ws + WS_CTRL_BYTES) + 4 * (size_t)row;
  uint32_t* h = (uint32_t*)((char*)ws + pct_hist_offset(gridDim.x)) + (size_t)row * PCT_BINS;
  if (threadIdx.x == 0) {
    st[0] = 0u;  // decided high bits
    st[1] = 0u;  // their mask
    st[2] = (uint32_t)m;  // 1-based rank within the matching values
    st[3] = 0u;
  }
  for (int i = threadIdx.x; i < PCT_BINS; i += blockDim.x) h[i] = 0u;
}

// grid (slices, rows); slice s of a row covers values [s*chunk, min(n, (s+1)*chunk))
template <bool V4>
__global__ __launch_bounds__(PCT_HNT) void pct_hist_kernel(const float* __restrict__ values,
                                                           int64_t n, int64_t chunk, int pass,
                                                           int rows, void* ws) {
  __shared__ uint32_t hist[PCT_HCOPIES][PCT_BINS];
  const int tid = threadIdx.x, copy = (tid / WAVE) % PCT_HCOPIES;
  const int row = blockIdx.y;
  const uint32_t* st = (const uint32_t*)((const char*)ws + WS_CTRL_BYTES) + 4 * (size_t)row;
  const uint32_t prefix = st[0], known = st[1];
  const int sh = pass == 0 ? 20 : (pass == 1 ? 10 : 0);
  const uint32_t nb = pass == 0 ? 2048u : 1024u;
  for (int i = tid; i < PCT_HCOPIES * PCT_BINS; i += PCT_HNT) (&hist[0][0])[i] = 0u;
  __syncthreads();
  const float* rowp = values + (size_t)row * (size_t)n;
  const int64_t lo = (int64_t)blockIdx.x * chunk, hi = lo + chunk < n ? lo + chunk : n;
  bool nan = false;
  auto count = [&](float v) {
    const uint32_t key = __float_as_uint(v) & 0x7FFFFFFFu;
    if (pass == 0 && key > 0x7F800000u) nan = true;
    if ((key & known) == prefix) atomicAdd(&hist[copy][(key >> sh) & (nb - 1)], 1u);
  };
  if constexpr (V4) {  // chunk and n are multiples of 4
    const float4* r4 = (const float4*)(rowp + lo);
    const int64_t n4 = (hi - lo) / 4;
    for (int64_t i = tid; i < n4; i += PCT_HNT) {
      const float4 v = r4[i];
      count(v.x);
      count(v.y);
      count(v.z);
      count(v.w);
    }
  } else {
    for (int64_t i = lo + tid; i < hi; i += PCT_HNT) count(rowp[i]);
  }
  if (nan) raise_error(ws, NP_DEVERR_NAN_SCORE);
  __syncthreads();
  uint32_t* h = (uint32_t*)((char*)ws + pct_hist_offset(rows)) + (size_t)row * PCT_BINS;
  for (int b = tid; b < (int)nb; b += PCT_HNT) {
    uint32_t c = 0u;
#pragma unroll
    for (int cp = 0; cp < PCT_HCOPIES; ++cp) c += hist[cp][b];
    if (c) atomicAdd(&h[b], c);
  }
}

// one workgroup per row: the digit of this pass that holds the rank
__global__ __launch_bounds__(PCT_NT) void pct_select_kernel(int pass, int rows, float* out,
                                                            void* ws) {
  __shared__ uint32_t scan[PCT_NT / WAVE + 1];
  __shared__ uint32_t sel[2];
  const int tid = threadIdx.x, row = blockIdx.x;
  uint32_t* st = (uint32_t*)((char*)ws + WS_CTRL_BYTES) + 4 * (size_t)row;
  uint32_t* h = (uint32_t*)((char*)ws + pct_hist_offset(rows)) + (size_t)row * PCT_BINS;
  const int sh = pass == 0 ? 20 : (pass == 1 ? 10 : 0);
  const int nb = pass == 0 ? 2048 : 1024;
  const uint32_t rank = st[2];
  uint32_t c[2];  // thread t owns bins 2t, 2t + 1
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int b = 2 * tid + j;
    c[j] = b < nb ? h[b] : 0u;
  }
  if (tid == 0) {  // a rank beyond the count (NaN rows only) keeps digit 0
    sel[0] = 0u;
    sel[1] = rank;
  }
  uint32_t tot;
  const uint32_t before = block_excl_scan<PCT_NT>(c[0] + c[1], scan, &tot);
  if (before < rank && rank <= before + c[0]) {
    sel[0] = 2 * tid;
    sel[1] = rank - before;
  } else if (before + c[0] < rank && rank <= before + c[0] + c[1]) {
    sel[0] = 2 * tid + 1;
    sel[1] = rank - before - c[0];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 2; ++j) h[2 * tid + j] = 0u;  // PCT_BINS = 2 * PCT_NT
  if (tid == 0) {
    const uint32_t prefix = st[0] | (sel[0] << sh);
    st[0] = prefix;
    st[1] |= (uint32_t)(nb - 1) << sh;
    st[2] = sel[1];
    if (pass == 2) out[row] = __uint_as_float(prefix);
  }
}

hipError_t launch_percentile(const float* values, int rows, int64_t n, int64_t m, float* out,
                             void* ws, size_t ws_bytes, hipStream_t stream) {
  // slices per row: about four workgroups per compute unit in all, each over
  // at least 32K values
  const int64_t want = ((int64_t)1024 + rows - 1) / rows;
  int64_t slices = std::min<int64_t>(want, (n + 32767) / 32768);
  if (slices > 65535) slices = 65535;
  if (slices >= 2 && ws_bytes >= percentile_ws_bytes(rows)) {
    int64_t chunk = (n + slices - 1) / slices;
    chunk = (chunk + 3) / 4 * 4;  // whole float4 vectors
    slices = (n + chunk - 1) / chunk;
    hipLaunchKernelGGL(pct_init_kernel, dim3(rows), dim3(256), 0, stream, m, ws);
    for (int pass = 0; pass < 3; ++pass) {
      if (n % 4 == 0)
        hipLaunchKernelGGL(pct_hist_kernel<true>, dim3((unsigned)slices, rows), dim3(PCT_HNT), 0,
                           stream, values, n, chunk, pass, rows, ws);
      else
        hipLaunchKernelGGL(pct_hist_kernel<false>, dim3((unsigned)slices, rows), dim3(PCT_HNT),
                           0, stream, values, n, chunk, pass, rows, ws);
      hipLaunchKernelGGL(pct_select_kernel, dim3(rows), dim3(PCT_NT), 0, stream, pass, rows, out,
                         ws);
    }
    return hipGetLastError();
  }
  if (n % 4 == 0)
    hipLaunchKernelGGL(percentile_kernel<true>, dim3(rows), dim3(PCT_NT), 0, stream, values, n,
                       m, out, ws);
  else
    hipLaunchKernelGGL(percentile_kernel<false>, dim3(rows), dim3(PCT_NT), 0, stream, values, n,
                       m, out, ws);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// eq. 1 as an active set
// ---------------------------------------------------------------------------
// One workgroup per row; thread t owns id words [t*WPT, t*WPT + WPT): it
// compares the word's 32 activations with the row's threshold, and a
// workgroup prefix sum over the words' popcounts places the ids in ascending
// order (the selection's layout).
template <int NT, int WPT, bool V4>
__global__ __launch_bounds__(NT) void threshold_active_kernel(
    const float* __restrict__ acts, const float* __restrict__ thr, uint32_t* __restrict__ mask,
    int32_t* __restrict__ active_ids, int32_t* __restrict__ counts, int F, int k, void* ws) {
  __shared__ uint32_t scan[NT / WAVE + 1];
  const int r = blockIdx.x, tid = threadIdx.x;
  const int W = (F + 31) / 32;
  const float T = thr[r];
  const float* row = acts + (size_t)r * F;
  uint32_t m[WPT], cnt = 0;
  bool nan = false;
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    const int word = tid * WPT + i;
    m[i] = 0u;
    if (word < W) {
      if (V4 && 32 * word + 32 <= F) {
        const float4* p = (const float4*)(row + 32 * word);
        float4 v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = p[j];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float e[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            nan |= e[c] != e[c];
            if (fabsf(e[c]) >= T) m[i] |= 1u << (4 * j + c);
          }
        }
      } else {
        for (int b = 0; b < 32 && 32 * word + b < F; ++b) {
          const float e = row[32 * word + b];
          nan |= e != e;
          if (fabsf(e) >= T) m[i] |= 1u << b;
        }
      }
      mask[(size_t)r * W + word] = m[i];
    }
    cnt += __builtin_popcount(m[i]);
  }
  if (nan) raise_error(ws, NP_DEVERR_NAN_SCORE);
  uint32_t tot;
  uint32_t pos = block_excl_scan<NT>(cnt, scan, &tot);
  int32_t* ids = active_ids + (size_t)r * k;
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    uint32_t bits = m[i];
    while (bits) {
      const int b = __builtin_ctz(bits);
      bits &= bits - 1;
      if (pos < (uint32_t)k) ids[pos] = 32 * (tid * WPT + i) + b;
      ++pos;
    }
  }
  if (tid == 0) {
    counts[r] = tot < (uint32_t)k ? (int32_t)tot : k;
    if (tot > (uint32_t)k) raise_error(ws, NP_DEVERR_OVERFLOW);
  }
}

hipError_t launch_threshold_active(const np_shape& s, const float* acts, int rows,
                                   const float* thr, uint32_t* mask, int32_t* active_ids,
                                   int32_t* active_counts, void* ws, hipStream_t stream) {
  const int words = (s.d_ffn + 31) / 32;
  const bool v4 = s.d_ffn % 4 == 0;
#define NP_THR_CASE(NT, W)                                                                     \
  do {                                                                                         \
    if (v4)                                                                                    \
      hipLaunchKernelGGL((threshold_active_kernel<NT, W, true>), dim3(rows), dim3(NT), 0,      \
                         stream, acts, thr, mask, active_ids, active_counts, s.d_ffn, s.k, ws); \
    else                                                                                       \
      hipLaunchKernelGGL((threshold_active_kernel<NT, W, false>), dim3(rows), dim3(NT), 0,     \
                         stream, acts, thr, mask, active_ids, active_counts, s.d_ffn, s.k, ws); \
  } while (0)
  if (words <= 256) NP_THR_CASE(256, 1);
  else if (words <= 512) NP_THR_CASE(512, 1);
  else if (words <= 1024) NP_THR_CASE(1024, 1);
  else NP_THR_CASE(1024, 2);
#undef NP_THR_CASE
  return hipGetLastError();
}

}  // namespace np
