// np_select.hip -- fixed-size active sets and the delta against the resident
// buffer (Sec. 3.4).  Both steps are small, latency-bound integer work: one
// 1024-thread workgroup per downstream layer, ids owned in 32-bit words so
// that set membership, ordering and compaction are bit operations, popcounts
// and workgroup prefix sums.  Both share the radix k-selection primitive of
// np_device.hpp (top-k of the scores; least-recently-used victims).
#include "np_device.hpp"

namespace np {

constexpr int SEL_NT = 1024;

// Order-preserving unsigned key of an fp32 score: larger score, larger key.
// -0.0 maps to the key of +0.0.  NaN maps to 0 (below every other key) and
// is reported through the error word.
__device__ inline uint32_t score_key(float f, bool* nan) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) {
    *nan = true;
    return 0u;
  }
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

template <int WPT>
__global__ __launch_bounds__(SEL_NT) void select_kernel(const float* __restrict__ scores,
                                                         uint32_t* __restrict__ mask,
                                                         int32_t* __restrict__ active_ids,
                                                         int F, int k, void* ws) {
  __shared__ uint32_t hist[4096];
  __shared__ uint32_t scan[SEL_NT / WAVE + 1];
  __shared__ uint32_t res[2];
  const int l = blockIdx.x, tid = threadIdx.x;
  const int words = (F + 31) / 32;
  const float* s = scores + (size_t)l * F;
  uint32_t key[WPT][32];
  bool nan = false;
#pragma unroll
  for (int w = 0; w < WPT; ++w) {
    const int word = tid * WPT + w;
#pragma unroll
    for (int b = 0; b < 32; ++b) {
      const int n = 32 * word + b;
      key[w][b] = (n < F) ? score_key(s[n], &nan) : 0u;
    }
  }
  if (nan) raise_error(ws, NP_DEVERR_NAN_SCORE);
  uint32_t sel[WPT];
  block_select_largest<SEL_NT, WPT>(key, (uint32_t)k, sel, hist, scan, res);
  uint32_t cnt = 0;
#pragma unroll
  for (int w = 0; w < WPT; ++w) cnt += __builtin_popcount(sel[w]);
  uint32_t tot;
  uint32_t pos = block_excl_scan<SEL_NT>(cnt, scan, &tot);
  int32_t* ids = active_ids + (size_t)l * k;
#pragma unroll
  for (int w = 0; w < WPT; ++w) {
    const int word = tid * WPT + w;
    if (word < words) mask[(size_t)l * words + word] = sel[w];
    uint32_t bits = sel[w];
    while (bits) {
      const int b = __builtin_ctz(bits);
      bits &= bits - 1;
      if (pos < (uint32_t)k) ids[pos] = 32 * word + b;
      ++pos;
    }
  }
}

// One workgroup per layer.  Thread t owns: actives j in [t*JPT, t*JPT+JPT),
// id words [t*WPT, t*WPT+WPT) and slot words [t*spt, t*spt+spt), so every
// list below comes out in ascending order from a prefix sum in thread order.
template <int WPT, int JPT>
__global__ __launch_bounds__(SEL_NT) void delta_kernel(int32_t token,
                                                        const int32_t* __restrict__ active_ids,
                                                        int32_t* __restrict__ slot_of,
                                                        int32_t* __restrict__ neuron_of,
                                                        int32_t* __restrict__ last_used,
                                                        np_delta_out out, int F, int C, int k,
                                                        int spt, void* ws) {
  __shared__ uint32_t amask[2048];  // active set, bit n of the layer
  __shared__ uint32_t smask[2048];  // slot pool: free slots, then victims' slots
  __shared__ uint32_t hist[4096];
  __shared__ uint32_t scan[SEL_NT / WAVE + 1];
  __shared__ uint32_t res[2];
  const int l = blockIdx.x, tid = threadIdx.x;
  const int idwords = (F + 31) / 32, slotwords = (C + 31) / 32;
  int32_t* P = slot_of + (size_t)l * F;
  int32_t* Q = neuron_of + (size_t)l * C;
  int32_t* U = last_used + (size_t)l * F;
  const int32_t* A = active_ids + (size_t)l * k;
  const size_t lo = (size_t)l * k;

  for (int i = tid; i < idwords; i += SEL_NT) amask[i] = 0;
  __syncthreads();

  // 1. hits and incoming rows, in active-list order
  int nj[JPT], pj[JPT];
  uint32_t hits = 0, incs = 0;
#pragma unroll
  for (int q = 0; q < JPT; ++q) {
    const int j = tid * JPT + q;
    nj[q] = -1;
    pj[q] = -1;
    if (j < k) {
      int n = A[j];
      if (n < 0 || n >= F) {  // not a neuron id: reported, counted as a miss
        raise_error(ws, NP_DEVERR_STATE);
        n = -1;
      }
      nj[q] = n;
      pj[q] = n >= 0 ? P[n] : -1;
      if (pj[q] >= C) {
        raise_error(ws, NP_DEVERR_STATE);
        pj[q] = -1;
      }
      if (n >= 0) atomicOr(&amask[n >> 5], 1u << (n & 31));
      if (pj[q] >= 0) ++hits;
      else ++incs;
    }
  }
  uint32_t tot;
  const uint32_t before = block_excl_scan<SEL_NT>(hits | (incs << 16), scan, &tot);
  const uint32_t nH = tot & 0xFFFFu, nI = tot >> 16;

  // 2. free slots (and a consistency check of the slot map)
  uint32_t nfree_local = 0;
  for (int q = 0; q < spt; ++q) {
    const int sw = tid * spt + q;
    if (sw >= slotwords) break;
    uint32_t bits = 0;
    for (int b = 0; b < 32; ++b) {
      const int sl = 32 * sw + b;
      if (sl >= C) break;
      const int qn = Q[sl];
      if (qn == -1) bits |= 1u << b;
      else if (qn < 0 || qn >= F || P[qn] != sl) raise_error(ws, NP_DEVERR_STATE);
    }
    smask[sw] = bits;
    nfree_local += __builtin_popcount(bits);
  }
  uint32_t nfree;
  (void)block_excl_scan<SEL_NT>(nfree_local, scan, &nfree);
  const uint32_t m = nI > nfree ? nI - nfree : 0u;

  // 3. victims: the m resident, non-active rows with the smallest
  //    (last_used, id) -- the largest keys ~last_used, ties to lower ids
  uint32_t vsel[WPT];
#pragma unroll
  for (int w = 0; w < WPT; ++w) vsel[w] = 0;
  if (m > 0) {
    uint32_t key[WPT][32];
#pragma unroll
    for (int w = 0; w < WPT; ++w) {
      const int word = tid * WPT + w;
#pragma unroll
      for (int b = 0; b < 32; ++b) {
        const int n = 32 * word + b;
        bool cand = false;
        if (n < F) {
          const int pn = P[n];
          cand = pn >= 0 && pn < C && !((amask[word] >> b) & 1u);
        }
        key[w][b] = cand ? ~(uint32_t)U[n] : 0u;
      }
    }
    block_select_largest<SEL_NT, WPT>(key, m, vsel, hist, scan, res);
    uint32_t cv = 0;
#pragma unroll
    for (int w = 0; w < WPT; ++w) cv += __builtin_popcount(vsel[w]);
    uint32_t vt;
    uint32_t vpos = block_excl_scan<SEL_NT>(cv, scan, &vt);
#pragma unroll
    for (int w = 0; w < WPT; ++w) {
      uint32_t bits = vsel[w];
      while (bits) {
        const int n = 32 * (tid * WPT + w) + __builtin_ctz(bits);
        bits &= bits - 1;
        const int old = P[n];
        if (old < 0 || old >= C || vpos >= (uint32_t)k) {  // only with a corrupted state
          raise_error(ws, NP_DEVERR_STATE);
          continue;
        }
        out.ev_ids[lo + vpos] = n;
        out.ev_slots[lo + vpos] = old;
        ++vpos;
        atomicOr(&smask[old >> 5], 1u << (old & 31));
      }
    }
  }
  __syncthreads();

  // 4. the slot pool in ascending order: its first nI slots go to the
  //    incoming rows (ascending ids)
  uint32_t cs = 0;
  for (int q = 0; q < spt; ++q) {
    const int sw = tid * spt + q;
    if (sw < slotwords) cs += __builtin_popcount(smask[sw]);
  }
  uint32_t st;
  uint32_t spos = block_excl_scan<SEL_NT>(cs, scan, &st);
  const uint32_t spos_total = st < nI ? st : nI;  // slots actually handed out
  for (int q = 0; q < spt; ++q) {
    const int sw = tid * spt + q;
    if (sw >= slotwords) break;
    uint32_t bits = smask[sw];
    while (bits && spos < nI) {
      const int b = __builtin_ctz(bits);
      bits &= bits - 1;
      out.in_slots[lo + spos] = 32 * sw + b;
      ++spos;
    }
  }

  // 5. victims release their slots
#pragma unroll
  for (int w = 0; w < WPT; ++w) {
    uint32_t bits = vsel[w];
    while (bits) {
      const int n = 32 * (tid * WPT + w) + __builtin_ctz(bits);
      bits &= bits - 1;
      const int old = P[n];
      if (old >= 0 && old < C) Q[old] = -1;
      P[n] = -1;
    }
  }
  __syncthreads();

  // 6. incoming rows take their slots; lists and last_used
  uint32_t hb = before & 0xFFFFu, ib = before >> 16;
#pragma unroll
  for (int q = 0; q < JPT; ++q) {
    const int j = tid * JPT + q;
    if (j < k) {
      const int n = nj[q];
      int slot;
      if (pj[q] >= 0) {
        slot = pj[q];
        out.hit_ids[lo + hb] = n;
        ++hb;
      } else {
        // the pool holds at least nI slots unless the state was corrupted
        slot = ib < spos_total ? out.in_slots[lo + ib] : -1;
        out.in_ids[lo + ib] = n;
        if (n >= 0 && slot >= 0 && slot < C) {
          P[n] = slot;
          Q[slot] = n;
        } else {
          raise_error(ws, NP_DEVERR_STATE);
          slot = -1;
        }
        ++ib;
      }
      if (n >= 0) U[n] = token;
      out.active_slots[lo + j] = slot;
    }
  }
  if (tid == 0) {
    out.counts[(size_t)l * 4 + 0] = (int32_t)nI;
    out.counts[(size_t)l * 4 + 1] = (int32_t)nH;
    out.counts[(size_t)l * 4 + 2] = (int32_t)m;
    out.counts[(size_t)l * 4 + 3] = (int32_t)(nI - m);
  }
}

__global__ void fill_state_kernel(int32_t* __restrict__ a, size_t na, int32_t* __restrict__ b,
                                  size_t nb, int32_t* __restrict__ c, size_t nc,
                                  int32_t* __restrict__ ctrl) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  const size_t i0 = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (size_t i = i0; i < na; i += stride) a[i] = -1;
  for (size_t i = i0; i < nb; i += stride) b[i] = -1;
  for (size_t i = i0; i < nc; i += stride) c[i] = -1;
  for (size_t i = i0; i < WS_CTRL_BYTES / 4; i += stride) ctrl[i] = 0;
}

hipError_t launch_fill_state(const np_shape& s, const np_state& st, void* ws,
                             hipStream_t stream) {
  const size_t nf = (size_t)s.layers * s.d_ffn, nc = (size_t)s.layers * s.capacity;
  hipLaunchKernelGGL(fill_state_kernel, dim3(1024), dim3(256), 0, stream, st.slot_of, nf,
                     st.neuron_of, nc, st.last_used, nf, (int32_t*)ws);
  return hipGetLastError();
}

hipError_t launch_select(const np_shape& s, const float* scores, uint32_t* mask,
                         int32_t* active_ids, void* ws, hipStream_t stream) {
  const int words = (s.d_ffn + 31) / 32;
  if (words <= SEL_NT)
    hipLaunchKernelGGL((select_kernel<1>), dim3(s.layers), dim3(SEL_NT), 0, stream, scores,
                       mask, active_ids, s.d_ffn, s.k, ws);
  else
    hipLaunchKernelGGL((select_kernel<2>), dim3(s.layers), dim3(SEL_NT), 0, stream, scores,
                       mask, active_ids, s.d_ffn, s.k, ws);
  return hipGetLastError();
}

template <int WPT>
static hipError_t delta_w(const np_shape& s, int32_t token, const int32_t* active_ids,
                          const np_state& st, const np_delta_out& out, void* ws,
                          hipStream_t stream) {
  const int slotwords = (s.capacity + 31) / 32;
  const int spt = (slotwords + SEL_NT - 1) / SEL_NT;
  const int jpt = (s.k + SEL_NT - 1) / SEL_NT;
#define NP_DELTA_CASE(J)                                                                      \
  hipLaunchKernelGGL((delta_kernel<WPT, J>), dim3(s.layers), dim3(SEL_NT), 0, stream, token,  \
                     active_ids, st.slot_of, st.neuron_of, st.last_used, out, s.d_ffn,        \
                     s.capacity, s.k, spt, ws)
  if (jpt <= 1) NP_DELTA_CASE(1);
  else if (jpt <= 2) NP_DELTA_CASE(2);
  else if (jpt <= 4) NP_DELTA_CASE(4);
  else NP_DELTA_CASE(8);
#undef NP_DELTA_CASE
  return hipGetLastError();
}

hipError_t launch_delta(const np_shape& s, int32_t token, const int32_t* active_ids,
                        const np_state& st, const np_delta_out& out, void* ws,
                        hipStream_t stream) {
  const int words = (s.d_ffn + 31) / 32;
  if (words <= SEL_NT) return delta_w<1>(s, token, active_ids, st, out, ws, stream);
  return delta_w<2>(s, token, active_ids, st, out, ws, stream);
}

}  // namespace np
