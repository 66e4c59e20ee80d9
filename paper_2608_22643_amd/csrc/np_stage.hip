// np_stage.hip -- moving incoming neuron records into their resident slots
// (Sec. 3.5: a record holds the gate, up and down^T rows of one neuron, so a
// single contiguous copy of 3d elements places all three; the scatter writes
// each record into the slot the delta assigned).  Pure data movement: HBM or
// host-link bound.  One workgroup copies one whole record per iteration with
// 16-byte vectors, all loads of a record issued before its stores; loads and
// stores carry the nontemporal hint (with write-back stores the step's first
// sparse-MLP calls paid for the written lines: 7B step 1755 -> 1861 tokens/s
// with the hint).
#include "np_device.hpp"

namespace np {

constexpr int STAGE_NT = 256;
constexpr int STAGE_UNROLL = 8;

__device__ inline void copy_record(uint4* __restrict__ dst, const uint4* __restrict__ src,
                                   int rec_vecs) {
  for (int v0 = threadIdx.x; v0 < rec_vecs; v0 += STAGE_NT * STAGE_UNROLL) {
    uint4 t[STAGE_UNROLL];
#pragma unroll
    for (int u = 0; u < STAGE_UNROLL; ++u) {
      const int v = v0 + u * STAGE_NT;
      if (v < rec_vecs) t[u] = load_nt(src + v);
    }
#pragma unroll
    for (int u = 0; u < STAGE_UNROLL; ++u) {
      const int v = v0 + u * STAGE_NT;
      if (v < rec_vecs) store_nt(dst + v, t[u]);
    }
  }
}

// Gather: the plan is np_delta's device output.  Records of layers
// [lb, le) are numbered layer by layer; workgroup b copies records
// b, b + gridDim.x, ...  The layers' counts are read in one round (thread t:
// layer lb + t, STAGE_NT layers at a time) and a prefix sum in LDS places
// each record.  Entries outside [0, F) x [0, C) raise NP_DEVERR_NOT_RESIDENT
// and are skipped.
__global__ __launch_bounds__(STAGE_NT) void stage_gather_kernel(
    const int32_t* __restrict__ counts, const int32_t* __restrict__ in_ids,
    const int32_t* __restrict__ in_slots, int k, int F, int C, int lb, int le,
    const uint4* __restrict__ storage, uint4* __restrict__ resident, int rec_vecs, void* ws) {
  __shared__ int pre[STAGE_NT + 1];  // records before layer base + i
  __shared__ uint32_t scan[STAGE_NT / WAVE + 1];
  const int G = gridDim.x, bid = blockIdx.x, tid = threadIdx.x;
  int done = 0;  // records of the layers before this block of layers
  for (int base = lb; base < le; base += STAGE_NT) {
    const int l = base + tid;
    int n = 0;
    if (l < le) {
      n = counts[(size_t)l * 4];
      if (n < 0 || n > k) {  // not a count np_delta can produce
        raise_error(ws, NP_DEVERR_STATE);
        n = n < 0 ? 0 : k;
      }
    }
    uint32_t tot;
    const uint32_t before = block_excl_scan<STAGE_NT>((uint32_t)n, scan, &tot);
    pre[tid] = (int)before;
    if (tid == 0) pre[STAGE_NT] = (int)tot;
    __syncthreads();
    const int nl = le - base < STAGE_NT ? le - base : STAGE_NT;
    for (int r = ((bid - done) % G + G) % G; r < (int)tot; r += G) {
      int lo = 0, hi = nl - 1;  // the layer i with pre[i] <= r < pre[i + 1]
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (pre[mid] <= r) lo = mid;
        else hi = mid - 1;
      }
      const int ll = base + lo, j = r - pre[lo];
      const int id = in_ids[(size_t)ll * k + j];
      const int slot = in_slots[(size_t)ll * k + j];
      if (id < 0 || id >= F || slot < 0 || slot >= C) {
        if (tid == 0) raise_error(ws, NP_DEVERR_NOT_RESIDENT);
        continue;
      }
      copy_record(resident + ((size_t)ll * C + slot) * rec_vecs,
                  storage + ((size_t)ll * F + id) * rec_vecs, rec_vecs);
    }
    done += (int)tot;
    __syncthreads();  // pre is rewritten by the next block of layers
  }
}

// Scatter: n landed records and their int32 destination rows (row = layer *
// C + slot, checked on the host when the records are packed; a row outside
// [0, n_rows) is skipped all the same, so no record lands outside the
// resident buffer).
__global__ __launch_bounds__(STAGE_NT) void stage_scatter_kernel(
    const uint4* __restrict__ landing, const int32_t* __restrict__ dst_rows, int n, int rec_vecs,
    uint4* __restrict__ resident, int n_rows) {
  for (int r = blockIdx.x; r < n; r += gridDim.x) {
    const int row = dst_rows[r];
    if (row < 0 || row >= n_rows) continue;
    copy_record(resident + (size_t)row * rec_vecs, landing + (size_t)r * rec_vecs, rec_vecs);
  }
}

hipError_t launch_stage_gather(const np_shape& s, const np_delta_out& out, int lb, int le,
                               const void* storage, void* resident, void* ws,
                               hipStream_t stream, bool host_storage) {
  const int rec_vecs = 3 * s.d_model * dtype_size(s.wdtype) / 16;
  int grid = 128 * (le - lb);
  // over the host link 256 workgroups keep enough records in flight (the
  // same rate as 2048 on the MI355X host) and leave the CUs to the MLPs
  // that run beside a side-stream gather
  if (grid > (host_storage ? 256 : 2048)) grid = host_storage ? 256 : 2048;
  if (grid < 64) grid = 64;
  hipLaunchKernelGGL(stage_gather_kernel, dim3(grid), dim3(STAGE_NT), 0, stream, out.counts,
                     out.in_ids, out.in_slots, s.k, s.d_ffn, s.capacity, lb, le,
                     (const uint4*)storage, (uint4*)resident, rec_vecs, ws);
  return hipGetLastError();
}

hipError_t launch_stage_scatter(const np_shape& s, const void* landing, const int32_t* rows,
                                int n_records, void* resident, hipStream_t stream) {
  const int rec_vecs = 3 * s.d_model * dtype_size(s.wdtype) / 16;
  int grid = n_records < 2048 ? n_records : 2048;
  if (grid < 1) return hipSuccess;
  hipLaunchKernelGGL(stage_scatter_kernel, dim3(grid), dim3(STAGE_NT), 0, stream,
                     (const uint4*)landing, rows, n_records, rec_vecs, (uint4*)resident,
                     s.layers * s.capacity);
  return hipGetLastError();
}

}  // namespace np
