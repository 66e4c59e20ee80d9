// np_select.hip -- fixed-size active sets and the delta against the resident
// buffer (Sec. 3.4).  Both steps are small, latency-bound integer work: one
// 1024-thread workgroup per downstream layer, ids owned in 32-bit words so
// that set membership, ordering and compaction are bit operations, popcounts
// and workgroup prefix sums.  Both share the radix k-selection primitive of
// np_device.hpp (top-k of the scores; least-recently-used victims).
#include <stdlib.h>

#include "np_device.hpp"

namespace np {

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

// Keys of thread tid's id words [tid*WPT, tid*WPT+WPT) of one layer's
// scores (0 past F).  Loads are unconditional (clamped index) so that all of
// them are in flight together; the range test only picks the key.  V4: the
// layer's scores are 16-byte aligned (F a multiple of 4) and read as float4.
template <int WPT, bool V4>
__device__ inline void load_score_keys(const float* __restrict__ s, int F, int tid,
                                       uint32_t (&key)[WPT][32], bool* nan) {
  if (32 * WPT * tid < F) {
#pragma unroll
    for (int w = 0; w < WPT; ++w) {
      const int word = tid * WPT + w;
      float v[32];
      if constexpr (V4) {
        const float4* s4 = reinterpret_cast<const float4*>(s);
        const int last = F / 4 - 1;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float4 q = s4[min(8 * word + i, last)];
          v[4 * i] = q.x;
          v[4 * i + 1] = q.y;
          v[4 * i + 2] = q.z;
          v[4 * i + 3] = q.w;
        }
      } else {
#pragma unroll
        for (int b = 0; b < 32; ++b) v[b] = s[min(32 * word + b, F - 1)];
      }
#pragma unroll
      for (int b = 0; b < 32; ++b) {
        const uint32_t kv = score_key(v[b], nan);
        key[w][b] = (32 * word + b < F) ? kv : 0u;
      }
    }
  } else {
#pragma unroll
    for (int w = 0; w < WPT; ++w)
#pragma unroll
      for (int b = 0; b < 32; ++b) key[w][b] = 0u;
  }
}

// The selected words of one layer out: the mask, and the ids in ascending
// order (a workgroup prefix sum of the words' popcounts) to `ids` and, when
// non-null, to `ids_lds` as well.
template <int NT, int WPT>
__device__ inline void write_selection(const uint32_t (&sel)[WPT], int tid, int words, int k,
                                       uint32_t* __restrict__ mask_l, int32_t* __restrict__ ids,
                                       int32_t* ids_lds, uint32_t* scan) {
  uint32_t cnt = 0;
#pragma unroll
  for (int w = 0; w < WPT; ++w) cnt += __builtin_popcount(sel[w]);
  uint32_t tot;
  uint32_t pos = block_excl_scan<NT>(cnt, scan, &tot);
#pragma unroll
  for (int w = 0; w < WPT; ++w) {
    const int word = tid * WPT + w;
    if (word < words) mask_l[word] = sel[w];
    uint32_t bits = sel[w];
    while (bits) {
      const int b = __builtin_ctz(bits);
      bits &= bits - 1;
      if (pos < (uint32_t)k) {
        ids[pos] = 32 * word + b;
        if (ids_lds) ids_lds[pos] = 32 * word + b;
      }
      ++pos;
    }
  }
}

// One workgroup of NT threads per layer; thread t owns id words
// [t*WPT, t*WPT+WPT).
template <int NT, int WPT, bool V4>
__global__ __launch_bounds__(NT) void select_kernel(const float* __restrict__ scores,
                                                    uint32_t* __restrict__ mask,
                                                    int32_t* __restrict__ active_ids, int F,
                                                    int k, void* ws) {
  __shared__ uint32_t hist[4096];
  __shared__ uint32_t scan[3 * (NT / WAVE) + 1];
  __shared__ uint32_t res[4];
  const int l = blockIdx.x, tid = threadIdx.x;
  const int words = (F + 31) / 32;
  uint32_t key[WPT][32];
  bool nan = false;
  load_score_keys<WPT, V4>(scores + (size_t)l * F, F, tid, key, &nan);
  if (nan) raise_error(ws, NP_DEVERR_NAN_SCORE);
  uint32_t sel[WPT];
  block_select_largest<NT, WPT>(key, (uint32_t)k, sel, hist, scan, res);
  write_selection<NT, WPT>(sel, tid, words, k, mask + (size_t)l * words,
                           active_ids + (size_t)l * k, nullptr, scan);
}

// The rest of a radix select over `n` candidate keys gathered in LDS (all
// nonzero and under `prefix`/`pmask`): 8-bit passes from bit `hi` down over
// a histogram of 256 words at hist[0..], the bin placed by wave 0 (lane L
// sums the 4 bins L-th from the top, a wave prefix sum finds the rem-th key).
// Ends as block_select_largest's passes do: `prefix` the k-th key and `rem`
// the keys equal to it still to take, or at a bin needed whole (prefix its
// smallest key, rem no limit).  Every thread calls it.
template <int NT>
__device__ inline void select_candidates(const uint32_t* cand, uint32_t n, uint32_t* hist,
                                         uint32_t* scan, uint32_t* res, int hi,
                                         uint32_t& prefix, uint32_t& pmask, uint32_t& rem) {
  constexpr int NW = NT / WAVE;
  const int tid = threadIdx.x, lane = tid & (WAVE - 1), w = tid / WAVE;
  while (hi >= 0) {
    const int nbits = hi + 1 < 8 ? hi + 1 : 8;
    const int shift = hi + 1 - nbits;
    const uint32_t nb = 1u << nbits;
    if ((uint32_t)tid < nb) hist[tid] = 0;
    __syncthreads();
    for (uint32_t c = tid; c < n; c += NT) {
      const uint32_t kv = cand[c];
      if ((kv & pmask) == prefix) atomicAdd(&hist[(kv >> shift) & (nb - 1)], 1u);
    }
    __syncthreads();
    if (w == 0) {
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
            res[2] = h == rem - c;
            break;
          }
          c += h;
        }
      }
    }
    __syncthreads();
    prefix |= res[0] << shift;
    pmask |= (nb - 1) << shift;
    rem = res[1];
    hi = shift - 1;
    const bool whole = res[2] != 0u && hi >= 0;
    __syncthreads();  // hist and res are reused
    if (whole) {
      uint32_t kmn = 0xFFFFFFFFu;
      for (uint32_t c = tid; c < n; c += NT) {
        const uint32_t kv = cand[c];
        if ((kv & pmask) == prefix && kv < kmn) kmn = kv;
      }
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        const uint32_t o = __shfl_xor(kmn, off, WAVE);
        kmn = o < kmn ? o : kmn;
      }
      if (lane == 0) scan[w] = kmn;
      __syncthreads();
      kmn = scan[0];
      for (int i = 1; i < NW; ++i) kmn = scan[i] < kmn ? scan[i] : kmn;
      __syncthreads();
      prefix = kmn;
      rem = 0xFFFFFFFFu;
      return;
    }
  }
}

// The k largest score keys of one layer (ties to the smaller id), as
// block_select_largest, starting from a hint: the previous token's k-th key
// and a window half-width, kept per layer in the workspace.  Scores change
// little from one token to the next, so the new k-th key usually lies in
// [key - half, key + half].  One pass counts the keys above the window and
// the keys in it; if the k-th key is inside (fewer than k above it, at least
// k above its lower end) and the window holds at most SEL_HINT_CAP keys,
// those keys go to LDS and the search finishes on them alone; otherwise the
// full radix select runs.  Either way the result is the same, and the hint
// is updated: the new k-th key, the window halved when it held many keys,
// quadrupled when the k-th key fell outside it.  hist: 4096 words of LDS.
constexpr uint32_t SEL_HINT_CAP = 4096 - 256;  // candidates kept after hist's first 256 words
constexpr uint32_t SEL_HINT_HALF0 = 1u << 20;  // first window half-width (fp32 keys: 0.125 at 1.0)

template <int NT>
__device__ inline void select_largest_hinted(const uint32_t (&key)[1][32], uint32_t kk,
                                             uint32_t (&sel)[1], uint32_t* hist, uint32_t* scan,
                                             uint32_t* res, uint32_t* hint) {
  constexpr int NW = NT / WAVE;
  const int tid = threadIdx.x, lane = tid & (WAVE - 1), w = tid / WAVE;
  const uint32_t hkey = hint ? hint[0] : 0u, hhalf = hint ? hint[1] : 0u;
  const uint32_t lo = hkey > hhalf ? hkey - hhalf : 1u;
  const uint32_t hi_w = hkey < 0xFFFFFFFFu - hhalf ? hkey + hhalf : 0xFFFFFFFFu;
  // nonzero keys, keys above the window, keys in it
  uint32_t nz = 0, above = 0, inside = 0;
#pragma unroll
  for (int b = 0; b < 32; ++b) {
    const uint32_t kv = key[0][b];
    nz += kv != 0u;
    above += kv > hi_w;
    inside += kv >= lo && kv <= hi_w;
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    nz += __shfl_xor(nz, off, WAVE);
    above += __shfl_xor(above, off, WAVE);
    inside += __shfl_xor(inside, off, WAVE);
  }
  if (lane == 0) {
    scan[w] = nz;
    scan[NW + w] = above;
    scan[2 * NW + w] = inside;
  }
  __syncthreads();
  nz = above = inside = 0;
  for (int i = 0; i < NW; ++i) {
    nz += scan[i];
    above += scan[NW + i];
    inside += scan[2 * NW + i];
  }
  __syncthreads();  // scan is reused below
  const bool use = hkey != 0u && hhalf != 0u && kk < nz && above < kk && kk <= above + inside &&
                   inside <= SEL_HINT_CAP;
  uint32_t prefix = 0, rem = 0;
  if (use) {
    // the window's keys, in LDS after hist's first 256 words
    uint32_t* cand = hist + 256;
    uint32_t mine = 0;
#pragma unroll
    for (int b = 0; b < 32; ++b) mine += key[0][b] >= lo && key[0][b] <= hi_w;
    uint32_t total;
    uint32_t at = block_excl_scan<NT>(mine, scan, &total);
#pragma unroll
    for (int b = 0; b < 32; ++b)
      if (key[0][b] >= lo && key[0][b] <= hi_w) cand[at++] = key[0][b];
    // bits above the highest one in which lo and hi_w differ are common to
    // every key of the window
    const uint32_t diff = lo ^ hi_w;
    const int hb = diff ? 31 - __builtin_clz(diff) : -1;
    const uint32_t low = hb >= 0 ? (uint32_t)((2ull << hb) - 1ull) : 0u;
    prefix = lo & ~low;
    uint32_t pmask = ~low;
    rem = kk - above;
    __syncthreads();  // cand complete
    select_candidates<NT>(cand, inside, hist, scan, res, hb, prefix, pmask, rem);
    sel[0] = 0;
  } else {
    uint32_t s0[1];
    block_select_largest<NT, 1>(key, kk, s0, hist, scan, res);
    sel[0] = s0[0];
  }
  uint32_t kth = 0;  // the k-th key: the smallest selected one
  if (use) {
    // take every key above the k-th and the first `rem` equal ones in id order
    uint32_t gt = 0, eq = 0;
#pragma unroll
    for (int b = 0; b < 32; ++b) {
      gt |= (key[0][b] > prefix ? 1u : 0u) << b;
      eq |= (key[0][b] == prefix ? 1u : 0u) << b;
    }
    uint32_t tot;
    uint32_t before = block_excl_scan<NT>(__builtin_popcount(eq), scan, &tot);
    while (eq && before < rem) {
      const uint32_t lowbit = eq & (0u - eq);
      gt |= lowbit;
      eq ^= lowbit;
      ++before;
    }
    sel[0] = gt;
    kth = prefix;
  } else if (hint && kk < nz) {
    uint32_t mn = 0xFFFFFFFFu;
#pragma unroll
    for (int b = 0; b < 32; ++b)
      if (((sel[0] >> b) & 1u) && key[0][b] < mn) mn = key[0][b];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const uint32_t o = __shfl_xor(mn, off, WAVE);
      mn = o < mn ? o : mn;
    }
    if (lane == 0) scan[w] = mn;
    __syncthreads();
    kth = scan[0];
    for (int i = 1; i < NW; ++i) kth = scan[i] < kth ? scan[i] : kth;
    __syncthreads();
  }
  if (hint && tid == 0) {
    uint32_t half = hhalf ? hhalf : SEL_HINT_HALF0;
    if (use) {
      if (inside > SEL_HINT_CAP / 4 && half > 1u) half >>= 1;
    } else if (hkey != 0u && hhalf != 0u) {
      half = half < (1u << 29) ? half << 2 : half;
    }
    hint[0] = kk < nz ? kth : 0u;
    hint[1] = half;
  }
}

// Limits of the fused selection + delta kernel (below): one id word per
// thread at 512 threads, and the layer's slot_of and neuron_of in LDS.
constexpr int SD_NT = 512;
constexpr int SD_MAX_F = 32 * SD_NT;  // 16384
constexpr int SD_MAX_C = 8192;
constexpr int SD_MAX_K = 4096;
constexpr int SD_PF = SD_MAX_F / SD_NT;  // slot_of loads per thread
constexpr int SD_QF = SD_MAX_C / SD_NT;  // neuron_of loads per thread

// The delta of one layer, run by all NT threads of its workgroup.  Thread t
// owns: actives j in [t*JPT, t*JPT+JPT), id words [t*WPT, t*WPT+WPT) and slot
// words [t*spt, t*spt+spt), so every list below comes out in ascending order
// from a prefix sum in thread order.
//   A: the layer's active ids (na of them, ascending); Pr, Qr: its slot_of
//   and neuron_of as they were at entry, read from global memory or from
//   copies in LDS; P, Q, U: the global slot_of, neuron_of and last_used,
//   which the delta updates (Pr and Qr may be P and Q themselves: no
//   restrict, and a thread reads an entry before any thread writes it).
//   LDS_STATE: Pr and Qr are in LDS, where the free-slot and residency scans
//   run as wave-wide passes (below); V4U: U's rows are 16-byte aligned (F a
//   multiple of 4) and the victim keys are read as int4; PRE_U: they were
//   read earlier, into upre (thread t: last_used of its id words).
//   amask, rmask: >= ceil(F/32) words, smask: >= ceil(C/32) words of LDS;
//   pool: >= na entries of LDS (it may share hist's storage: it is written
//   only after the last use of hist).
// Every global gather of a phase is issued unconditionally (clamped index)
// so that the phase costs one memory round trip, not one per element.
template <int NT, int WPT, int JPT, bool LDS_STATE, bool V4U, bool PRE_U>
__device__ __attribute__((always_inline)) inline void delta_layer(int l, int32_t token, const int32_t* A, int na, bool bad_count,
                                   const int32_t* Pr, const int32_t* Qr, int32_t* P, int32_t* Q,
                                   int32_t* U, const uint32_t (&upre)[WPT][32],
                                   const np_delta_out& out, int F, int C, int k, int spt,
                                   void* ws, uint32_t* amask, uint32_t* smask, uint32_t* rmask,
                                   uint32_t* hist, int32_t* pool, uint32_t* scan,
                                   uint32_t* res) {
  const int tid = threadIdx.x, lane = tid & (WAVE - 1), wv = tid / WAVE;
  const int idwords = (F + 31) / 32, slotwords = (C + 31) / 32;
  const size_t lo = (size_t)l * k;

  for (int i = tid; i < idwords; i += NT) {
    amask[i] = 0;
    rmask[i] = 0;
  }
  __syncthreads();

  // 1. hits and incoming rows, in active-list order
  int nj[JPT], pj[JPT];
  uint32_t hits = 0, incs = 0, bad = 0;
#pragma unroll
  for (int q = 0; q < JPT; ++q) nj[q] = A[min(tid * JPT + q, na > 0 ? na - 1 : 0)];
#pragma unroll
  for (int q = 0; q < JPT; ++q) {
    const bool ok = nj[q] >= 0 && nj[q] < F;  // else not a neuron id: counted as a miss
    if (tid * JPT + q < na) bad |= !ok;
    if (!ok) nj[q] = -1;
    pj[q] = Pr[nj[q] >= 0 ? nj[q] : 0];
  }
  int qb[JPT];  // a hit's slot must hold it
#pragma unroll
  for (int q = 0; q < JPT; ++q) qb[q] = Qr[(pj[q] >= 0 && pj[q] < C) ? pj[q] : 0];
#pragma unroll
  for (int q = 0; q < JPT; ++q) {
    const int j = tid * JPT + q;
    if (nj[q] < 0 || pj[q] >= C) {
      bad |= (j < na) & (pj[q] >= C) & (nj[q] >= 0);
      pj[q] = -1;
    }
    if (pj[q] >= 0 && qb[q] != nj[q]) {
      bad |= j < na;
      pj[q] = -1;
    }
    if (j < na) {
      if (nj[q] >= 0) atomicOr(&amask[nj[q] >> 5], 1u << (nj[q] & 31));
      if (pj[q] >= 0) ++hits;
      else ++incs;
    }
  }
  uint32_t tot;
  const uint32_t before = block_excl_scan<NT>(hits | (incs << 16), scan, &tot);
  const uint32_t nH = tot & 0xFFFFu, nI = tot >> 16;

  // 2. free slots and resident rows, and a consistency check of the slot
  //    map: a used slot's neuron must map back to it
  uint32_t nfree_local = 0;
  if constexpr (LDS_STATE) {
    // wave-wide passes over the slots: lane i takes slot base + i of 64
    // consecutive ones, a ballot gives two words of free slots; a used
    // slot's neuron must map back to it.
    static_assert(NT == SD_NT, "the LDS path runs at SD_NT threads");
    constexpr int NS = SD_MAX_C / SD_NT;
    // the ballots stay in registers: lane 2j + h keeps word h of pass j and
    // stores it after the loop.  A used slot whose neuron maps back to it
    // marks that neuron resident.
    uint32_t word = 0;
    const int passes = (C - wv * WAVE + NT - 1) / NT;  // this wave's passes (<= NS)
    for (int j = 0; j < passes; ++j) {
      const int sl = wv * WAVE + j * NT + lane;
      const int qv = Qr[min(sl, C - 1)];
      const int back = Pr[(uint32_t)qv < (uint32_t)F ? qv : 0];
      const bool in = sl < C, used = in & (qv != -1);
      const bool pair = ((uint32_t)qv < (uint32_t)F) & (back == sl);
      bad |= used & !pair;
      if (used & pair) atomicOr(&rmask[qv >> 5], 1u << (qv & 31));
      const uint64_t fm = __ballot(in & (qv == -1));
      word = lane == 2 * j ? (uint32_t)fm : (lane == 2 * j + 1 ? (uint32_t)(fm >> 32) : word);
      nfree_local += lane == 0 ? __popcll(fm) : 0;
    }
    {
      const int wi = 2 * wv + (NT / 32) * (lane / 2) + (lane & 1);
      if (lane < 2 * NS && wi < slotwords) smask[wi] = word;
    }
  } else
  for (int q = 0; q < spt; ++q) {
    const int sw = tid * spt + q;
    if (sw >= slotwords) break;
    int qn[32];
#pragma unroll
    for (int b = 0; b < 32; ++b) qn[b] = Qr[min(32 * sw + b, C - 1)];
    uint32_t bits = 0;
#pragma unroll
    for (int h = 0; h < 2; ++h) {  // halves: 16 back-gathers in flight
      int back[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int qv = qn[16 * h + i];
        back[i] = Pr[(qv >= 0 && qv < F) ? qv : 0];
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int b = 16 * h + i, sl = 32 * sw + b, qv = qn[b];
        if (sl < C) {
          if (qv == -1) {
            bits |= 1u << b;
          } else if (qv < 0 || qv >= F || back[i] != sl) {
            bad = 1;
          } else {
            atomicOr(&rmask[qv >> 5], 1u << (qv & 31));
          }
        }
      }
    }
    smask[sw] = bits;
    nfree_local += __builtin_popcount(bits);
  }
  uint32_t nfree;
  (void)block_excl_scan<NT>(nfree_local, scan, &nfree);  // its barriers publish rmask
  const uint32_t m = nI > nfree ? nI - nfree : 0u;

  // 3. victims: the m resident, non-active rows with the smallest
  //    (last_used, id) -- the largest keys ~last_used, ties to lower ids.
  //    Each victim leaves the slot map here: its slot joins the pool.
  uint32_t vsel[WPT];
#pragma unroll
  for (int w = 0; w < WPT; ++w) vsel[w] = 0;
  if (m > 0) {
    uint32_t key[WPT][32];
    if (32 * WPT * tid < F) {
#pragma unroll
      for (int w = 0; w < WPT; ++w) {
        const int word = tid * WPT + w;
        if constexpr (PRE_U) {
#pragma unroll
          for (int b = 0; b < 32; ++b) key[w][b] = upre[w][b];
        } else if constexpr (V4U) {
          const int4* u4 = reinterpret_cast<const int4*>(U);
          const int last = F / 4 - 1;
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const int4 q = u4[min(8 * word + i, last)];
            key[w][4 * i] = (uint32_t)q.x;
            key[w][4 * i + 1] = (uint32_t)q.y;
            key[w][4 * i + 2] = (uint32_t)q.z;
            key[w][4 * i + 3] = (uint32_t)q.w;
          }
        } else {
#pragma unroll
          for (int b = 0; b < 32; ++b) key[w][b] = (uint32_t)U[min(32 * word + b, F - 1)];
        }
        // resident, not active, and inside the layer (rmask has no bits past F)
        const uint32_t cm = word < idwords ? (rmask[word] & ~amask[word]) : 0u;
#pragma unroll
        for (int b = 0; b < 32; ++b) key[w][b] = ((cm >> b) & 1u) ? ~key[w][b] : 0u;
      }
    } else {
#pragma unroll
      for (int w = 0; w < WPT; ++w)
#pragma unroll
        for (int b = 0; b < 32; ++b) key[w][b] = 0u;
    }
    block_select_largest<NT, WPT>(key, m, vsel, hist, scan, res);
    uint32_t cv = 0;
#pragma unroll
    for (int w = 0; w < WPT; ++w) cv += __builtin_popcount(vsel[w]);
    uint32_t vt;
    uint32_t vpos = block_excl_scan<NT>(cv, scan, &vt);
#pragma unroll
    for (int w = 0; w < WPT; ++w) {
      if (!vsel[w]) continue;
      const int word = tid * WPT + w;
      if constexpr (LDS_STATE) {  // LDS: only the victims' entries, one by one
        uint32_t bits = vsel[w];
        while (bits) {
          const int b = __builtin_ctz(bits);
          bits &= bits - 1;
          const int n = 32 * word + b, old = Pr[n];
          if (old < 0 || old >= C || vpos >= (uint32_t)k) {  // only with a corrupted state
            bad = 1;
            continue;
          }
          out.ev_ids[lo + vpos] = n;
          out.ev_slots[lo + vpos] = old;
          ++vpos;
          atomicOr(&smask[old >> 5], 1u << (old & 31));
          Q[old] = -1;
          P[n] = -1;
        }
        continue;
      }
      int pn[32];
#pragma unroll
      for (int b = 0; b < 32; ++b) pn[b] = Pr[min(32 * word + b, F - 1)];
#pragma unroll
      for (int b = 0; b < 32; ++b) {
        if (!((vsel[w] >> b) & 1u)) continue;
        const int n = 32 * word + b, old = pn[b];
        if (old < 0 || old >= C || vpos >= (uint32_t)k) {  // only with a corrupted state
          bad = 1;
          continue;
        }
        out.ev_ids[lo + vpos] = n;
        out.ev_slots[lo + vpos] = old;
        ++vpos;
        atomicOr(&smask[old >> 5], 1u << (old & 31));
        Q[old] = -1;
        P[n] = -1;
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
  uint32_t spos = block_excl_scan<NT>(cs, scan, &st);
  const uint32_t spos_total = st < nI ? st : nI;  // slots actually handed out
  for (int q = 0; q < spt; ++q) {
    const int sw = tid * spt + q;
    if (sw >= slotwords) break;
    uint32_t bits = smask[sw];
    while (bits && spos < nI) {
      const int b = __builtin_ctz(bits);
      bits &= bits - 1;
      out.in_slots[lo + spos] = 32 * sw + b;
      pool[spos] = 32 * sw + b;
      ++spos;
    }
  }
  __syncthreads();

  // 5. incoming rows take their slots; lists and last_used
  uint32_t hb = before & 0xFFFFu, ib = before >> 16;
#pragma unroll
  for (int q = 0; q < JPT; ++q) {
    const int j = tid * JPT + q;
    if (j < na) {
      const int n = nj[q];
      int slot;
      if (pj[q] >= 0) {
        slot = pj[q];
        out.hit_ids[lo + hb] = n;
        ++hb;
      } else {
        // the pool holds at least nI slots unless the state was corrupted
        slot = ib < spos_total ? pool[ib] : -1;
        out.in_ids[lo + ib] = n;
        if (n >= 0 && slot >= 0 && slot < C) {
          P[n] = slot;
          Q[slot] = n;
        } else {
          bad = 1;
          slot = -1;
        }
        ++ib;
      }
      if (n >= 0) U[n] = token;
      out.active_slots[lo + j] = slot;
    }
  }
  if (bad || (bad_count && tid == 0)) raise_error(ws, NP_DEVERR_STATE);
  if (tid == 0) {
    out.counts[(size_t)l * 4 + 0] = (int32_t)nI;
    out.counts[(size_t)l * 4 + 1] = (int32_t)nH;
    out.counts[(size_t)l * 4 + 2] = (int32_t)m;
    out.counts[(size_t)l * 4 + 3] = (int32_t)(nI - m);
  }
}

// np_delta: one workgroup per layer, the state read from global memory.
template <int NT, int WPT, int JPT>
__global__ __launch_bounds__(NT) void delta_kernel(int32_t token,
                                                   const int32_t* __restrict__ active_ids,
                                                   int32_t* __restrict__ slot_of,
                                                   int32_t* __restrict__ neuron_of,
                                                   int32_t* __restrict__ last_used,
                                                   np_delta_out out, int F, int C, int k,
                                                   int spt, void* ws,
                                                   const int32_t* __restrict__ counts) {
  __shared__ uint32_t amask[2048];  // active set, bit n of the layer
  __shared__ uint32_t smask[2048];  // slot pool: free slots, then victims' slots
  __shared__ uint32_t rmask[2048];  // resident rows (neurons held by some slot)
  __shared__ uint32_t hist[4096];
  __shared__ int32_t pool[8192];    // the first nI pool slots, ascending
  __shared__ uint32_t scan[3 * (NT / WAVE) + 1];
  __shared__ uint32_t res[4];
  const int l = blockIdx.x;
  if (token == NP_TOKEN_AUTO) token = *(const int32_t*)((const char*)ws + WS_TOKEN);
  int32_t* P = slot_of + (size_t)l * F;
  int32_t* Q = neuron_of + (size_t)l * C;
  // active neurons of this layer: k, or a device count in [0, k]
  int na = k;
  bool bad_count = false;
  if (counts) {
    na = counts[l];
    if (na < 0 || na > k) {
      bad_count = true;
      na = na < 0 ? 0 : k;
    }
  }
  const uint32_t none[WPT][32] = {};
  delta_layer<NT, WPT, JPT, false, false, false>(l, token, active_ids + (size_t)l * k, na,
                                                 bad_count, P, Q, P, Q, last_used + (size_t)l * F,
                                                 none, out, F, C, k, spt, ws, amask, smask, rmask,
                                                 hist, pool, scan, res);
}

// np_select followed by np_delta in one workgroup per layer.  At entry every
// thread issues all of its loads at once: the scores of its id word (the
// selection keys), the last_used values of the same word (the victim keys)
// and a share of the layer's slot_of and neuron_of, which go to LDS; the delta then finds every slot and back-reference there instead
// of in global memory, scans the slots and neurons wave by wave, and needs no
// second launch.  For F <= SD_MAX_F, C <= SD_MAX_C and
// k <= SD_MAX_K (one id word per thread at 512 threads); the slot pool of the
// delta shares the selection's histogram.

template <int JPT, bool V4>
__global__ __launch_bounds__(SD_NT) void select_delta_kernel(
    const float* __restrict__ scores, uint32_t* __restrict__ mask,
    int32_t* __restrict__ active_ids, int32_t token, int32_t* __restrict__ slot_of,
    int32_t* __restrict__ neuron_of, int32_t* __restrict__ last_used, np_delta_out out, int F,
    int C, int k, void* ws) {
  constexpr int NT = SD_NT;
  __shared__ __attribute__((aligned(16))) int32_t Ps[SD_MAX_F];  // slot_of of the layer at entry
  __shared__ int32_t Qs[SD_MAX_C];  // neuron_of of the layer at entry
  __shared__ int32_t ids_s[SD_MAX_K];
  __shared__ uint32_t amask[SD_MAX_F / 32], rmask[SD_MAX_F / 32], smask[SD_MAX_C / 32];
  __shared__ uint32_t hist[4096];  // both selections; then the delta's slot pool
  __shared__ uint32_t scan[3 * (NT / WAVE) + 1];
  __shared__ uint32_t res[4];
  const int l = blockIdx.x, tid = threadIdx.x;
  if (token == NP_TOKEN_AUTO) token = *(const int32_t*)((const char*)ws + WS_TOKEN);
  const int words = (F + 31) / 32;
  int32_t* P = slot_of + (size_t)l * F;
  int32_t* Q = neuron_of + (size_t)l * C;
  int32_t* U = last_used + (size_t)l * F;
  // all loads first: slot_of (int4 when its rows are 16-byte aligned), the
  // selection keys, neuron_of and the victim keys' last_used values.  Loads
  // complete in order: slot_of goes to LDS as soon as it is in, the
  // selection waits only for the keys, and neuron_of goes to LDS after it.
  // (A clamped index loads and stores the last entry again, with the same
  // value: the loops have no branch, so they unroll and stay in registers.)
  constexpr int PV = V4 ? SD_PF / 4 : SD_PF;
  int4 pv4[V4 ? PV : 1];
  int pv1[V4 ? 1 : PV];
  if constexpr (V4) {
    const int4* P4 = reinterpret_cast<const int4*>(P);
#pragma unroll
    for (int i = 0; i < PV; ++i) pv4[i] = P4[min(tid + NT * i, F / 4 - 1)];
  } else {
#pragma unroll
    for (int i = 0; i < PV; ++i) pv1[i] = P[min(tid + NT * i, F - 1)];
  }
  uint32_t key[1][32];
  bool nan = false;
  load_score_keys<1, V4>(scores + (size_t)l * F, F, tid, key, &nan);
  int qv[SD_QF];
#pragma unroll
  for (int i = 0; i < SD_QF; ++i) qv[i] = Q[min(tid + NT * i, C - 1)];
  uint32_t ukey[1][32] = {};  // with unaligned rows the delta reads them itself
  if constexpr (V4) {
    const int4* u4 = reinterpret_cast<const int4*>(U);
    const int last = F / 4 - 1;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int4 q = u4[min(8 * tid + i, last)];
      ukey[0][4 * i] = (uint32_t)q.x;
      ukey[0][4 * i + 1] = (uint32_t)q.y;
      ukey[0][4 * i + 2] = (uint32_t)q.z;
      ukey[0][4 * i + 3] = (uint32_t)q.w;
    }
  }
  if constexpr (V4) {
#pragma unroll
    for (int i = 0; i < PV; ++i)
      reinterpret_cast<int4*>(Ps)[min(tid + NT * i, F / 4 - 1)] = pv4[i];
  } else {
#pragma unroll
    for (int i = 0; i < PV; ++i) Ps[min(tid + NT * i, F - 1)] = pv1[i];
  }
  if (nan) raise_error(ws, NP_DEVERR_NAN_SCORE);
  uint32_t sel[1];
  uint32_t* hint = l < WS_SEL_HINT_LAYERS ? (uint32_t*)((char*)ws + WS_SEL_HINT) + 2 * l : nullptr;
  select_largest_hinted<NT>(key, (uint32_t)k, sel, hist, scan, res, hint);
#pragma unroll
  for (int i = 0; i < SD_QF; ++i) Qs[min(tid + NT * i, C - 1)] = qv[i];
  write_selection<NT, 1>(sel, tid, words, k, mask + (size_t)l * words,
                         active_ids + (size_t)l * k, ids_s, scan);
  __syncthreads();  // ids_s, Ps and Qs complete
  delta_layer<NT, 1, JPT, true, V4, V4>(l, token, ids_s, k, false, Ps, Qs, P, Q, U, ukey, out, F,
                                        C, k, 1, ws, amask, smask, rmask, hist, (int32_t*)hist,
                                        scan, res);
}

// Centroid choice and the intersected active set (Sec. 3.3-3.4), one
// workgroup per layer.  Waves 0 and 1 take the argmax of the layer's gate and
// up heads over the K logits (lane c reads c, c+64, ...; a NaN never wins and
// sets the error bit; equal values go to the smaller index).  Then thread t
// owns id words [t*WPT, t*WPT+WPT) of the AND of the two chosen masks, and a
// workgroup prefix sum places its ids in ascending order.
template <int NT, int WPT>
__global__ __launch_bounds__(NT) void centroid_active_kernel(
    const float* __restrict__ logits, const uint32_t* __restrict__ bank,
    int32_t* __restrict__ cids, uint32_t* __restrict__ mask, int32_t* __restrict__ active_ids,
    int32_t* __restrict__ counts, int L, int F, int K, int k, void* ws) {
  __shared__ int chosen[2];
  __shared__ uint32_t scan[NT / WAVE + 1];
  const int l = blockIdx.x, tid = threadIdx.x, lane = tid & (WAVE - 1), w = tid / WAVE;
  if (w < 2) {
    const int h = w * L + l;
    const float* lg = logits + (size_t)h * K;
    float best = 0.f;
    int bi = K;  // K: nothing seen yet
    bool nan = false;
    for (int c = lane; c < K; c += WAVE) {
      const float v = lg[c];
      if (v != v) {
        nan = true;
        continue;
      }
      if (bi == K || v > best) {  // ascending c: a lane keeps its first maximum
        best = v;
        bi = c;
      }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const float ob = __shfl_xor(best, off, WAVE);
      const int oi = __shfl_xor(bi, off, WAVE);
      if (oi != K && (bi == K || ob > best || (ob == best && oi < bi))) {
        best = ob;
        bi = oi;
      }
    }
    if (nan) raise_error(ws, NP_DEVERR_NAN_SCORE);
    if (lane == 0) {
      if (bi == K) bi = 0;  // every logit NaN: reported above
      chosen[w] = bi;
      cids[h] = bi;
    }
  }
  __syncthreads();
  const int W = (F + 31) / 32;
  const uint32_t* g = bank + ((size_t)l * K + chosen[0]) * W;
  const uint32_t* u = bank + (((size_t)L + l) * K + chosen[1]) * W;
  uint32_t m[WPT], cnt = 0;
#pragma unroll
  for (int i = 0; i < WPT; ++i) {
    const int word = tid * WPT + i;
    m[i] = word < W ? (g[word] & u[word]) : 0u;
    if (word == W - 1 && (F & 31)) m[i] &= (1u << (F & 31)) - 1u;
    if (word < W) mask[(size_t)l * W + word] = m[i];
    cnt += __builtin_popcount(m[i]);
  }
  uint32_t tot;
  uint32_t pos = block_excl_scan<NT>(cnt, scan, &tot);
  int32_t* ids = active_ids + (size_t)l * k;
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
    counts[l] = tot < (uint32_t)k ? (int32_t)tot : k;
    if (tot > (uint32_t)k) raise_error(ws, NP_DEVERR_OVERFLOW);
  }
}

hipError_t launch_centroid_active(const np_shape& s, const np_centroid_model& m,
                                  const float* logits, int32_t* centroid_ids, uint32_t* mask,
                                  int32_t* active_ids, int32_t* active_counts, void* ws,
                                  hipStream_t stream) {
  const int words = (s.d_ffn + 31) / 32;
#define NP_CENTROID_CASE(NT, W)                                                            \
  hipLaunchKernelGGL((centroid_active_kernel<NT, W>), dim3(s.layers), dim3(NT), 0, stream, \
                     logits, m.bank, centroid_ids, mask, active_ids, active_counts,         \
                     s.layers, s.d_ffn, m.n_centroids, s.k, ws)
  if (words <= 256) NP_CENTROID_CASE(256, 1);
  else if (words <= 512) NP_CENTROID_CASE(512, 1);
  else if (words <= 1024) NP_CENTROID_CASE(1024, 1);
  else NP_CENTROID_CASE(1024, 2);
#undef NP_CENTROID_CASE
  return hipGetLastError();
}

// Advances np_delta's step counter (NP_TOKEN_AUTO) once the delta is done.
__global__ void token_advance_kernel(void* ws) {
  if (threadIdx.x == 0) *(int32_t*)((char*)ws + WS_TOKEN) += 1;
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
  const bool v4 = s.d_ffn % 4 == 0;
#define NP_SELECT_CASE(NT, W)                                                                \
  do {                                                                                       \
    if (v4)                                                                                  \
      hipLaunchKernelGGL((select_kernel<NT, W, true>), dim3(s.layers), dim3(NT), 0, stream,  \
                         scores, mask, active_ids, s.d_ffn, s.k, ws);                        \
    else                                                                                     \
      hipLaunchKernelGGL((select_kernel<NT, W, false>), dim3(s.layers), dim3(NT), 0, stream, \
                         scores, mask, active_ids, s.d_ffn, s.k, ws);                        \
  } while (0)
  if (words <= 256) NP_SELECT_CASE(256, 1);
  else if (words <= 512) NP_SELECT_CASE(512, 1);
  else if (words <= 1024) NP_SELECT_CASE(1024, 1);
  else NP_SELECT_CASE(1024, 2);
#undef NP_SELECT_CASE
  return hipGetLastError();
}

template <int NT, int WPT>
static hipError_t delta_w(const np_shape& s, int32_t token, const int32_t* active_ids,
                          const np_state& st, const np_delta_out& out, void* ws,
                          hipStream_t stream, const int32_t* counts) {
  const int slotwords = (s.capacity + 31) / 32;
  const int spt = (slotwords + NT - 1) / NT;
  const int jpt = (s.k + NT - 1) / NT;
#define NP_DELTA_CASE(J)                                                                      \
  hipLaunchKernelGGL((delta_kernel<NT, WPT, J>), dim3(s.layers), dim3(NT), 0, stream, token,  \
                     active_ids, st.slot_of, st.neuron_of, st.last_used, out, s.d_ffn,        \
                     s.capacity, s.k, spt, ws, counts)
  if (jpt <= 1) NP_DELTA_CASE(1);
  else if (jpt <= 2) NP_DELTA_CASE(2);
  else if (jpt <= 4) NP_DELTA_CASE(4);
  else NP_DELTA_CASE(8);
#undef NP_DELTA_CASE
  return hipGetLastError();
}

hipError_t launch_delta(const np_shape& s, int32_t token, const int32_t* active_ids,
                        const np_state& st, const np_delta_out& out, void* ws,
                        hipStream_t stream, const int32_t* counts) {
  // 512 threads while every thread owns one id word and at most 4 actives
  const int words = (s.d_ffn + 31) / 32;
  hipError_t e;
  if (words <= 512 && s.k <= 2048) e = delta_w<512, 1>(s, token, active_ids, st, out, ws, stream, counts);
  else if (words <= 1024) e = delta_w<1024, 1>(s, token, active_ids, st, out, ws, stream, counts);
  else e = delta_w<1024, 2>(s, token, active_ids, st, out, ws, stream, counts);
  if (e != hipSuccess || token != NP_TOKEN_AUTO) return e;
  hipLaunchKernelGGL(token_advance_kernel, dim3(1), dim3(64), 0, stream, ws);
  return hipGetLastError();
}

// np_select then np_delta: the fused kernel where the layer fits it (unless
// NP_SELECT_DELTA_FUSED=0), else the two kernels.
hipError_t launch_select_delta(const np_shape& s, int32_t token, const float* scores,
                               uint32_t* mask, int32_t* active_ids, const np_state& st,
                               const np_delta_out& out, void* ws, hipStream_t stream) {
  const char* env = getenv("NP_SELECT_DELTA_FUSED");
  const bool fused = !(env && env[0] == '0') && s.d_ffn <= SD_MAX_F &&
                     s.capacity <= SD_MAX_C && s.k <= SD_MAX_K;
  if (!fused) {
    hipError_t e = launch_select(s, scores, mask, active_ids, ws, stream);
    if (e != hipSuccess) return e;
    return launch_delta(s, token, active_ids, st, out, ws, stream, nullptr);
  }
  const bool v4 = s.d_ffn % 4 == 0;
  const int jpt = (s.k + SD_NT - 1) / SD_NT;
#define NP_SD_CASE(J)                                                                            do {                                                                                             if (v4)                                                                                          hipLaunchKernelGGL((select_delta_kernel<J, true>), dim3(s.layers), dim3(SD_NT), 0,                                stream, scores, mask, active_ids, token, st.slot_of, st.neuron_of,                             st.last_used, out, s.d_ffn, s.capacity, s.k, ws);                         else                                                                                             hipLaunchKernelGGL((select_delta_kernel<J, false>), dim3(s.layers), dim3(SD_NT), 0,                               stream, scores, mask, active_ids, token, st.slot_of, st.neuron_of,                             st.last_used, out, s.d_ffn, s.capacity, s.k, ws);                       } while (0)
  if (jpt <= 1) NP_SD_CASE(1);
  else if (jpt <= 2) NP_SD_CASE(2);
  else if (jpt <= 4) NP_SD_CASE(4);
  else NP_SD_CASE(8);
#undef NP_SD_CASE
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || token != NP_TOKEN_AUTO) return e;
  hipLaunchKernelGGL(token_advance_kernel, dim3(1), dim3(64), 0, stream, ws);
  return hipGetLastError();
}

}  // namespace np
