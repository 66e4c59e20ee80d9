// np_internal.hpp -- definitions shared by the HIP kernels and the host side
// of libneuroprefetch (workspace layout, launch helpers, device utilities).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "neuroprefetch.h"

namespace np {

// ---------------------------------------------------------------------------
// Device workspace layout (dev_ws).  Offsets are multiples of 256 bytes.
//   [0, 4096)            control block
//       +0    int32  sticky error word (NP_DEVERR_* bits)
//       +64   int32  np_delta step counter (NP_TOKEN_AUTO)
//       +256  int32  sparse-MLP grid barrier: arrivals of the current call
//       +384  int32  sparse-MLP grid barrier: generation (calls completed)
//   [4096, +L'*r*4)      predictor intermediate z, fp32 [L'][r]
//   [.., +MLP_MAX_WG*ceil16(d)*4) sparse-MLP per-workgroup partial sums, fp32
// ---------------------------------------------------------------------------
constexpr size_t WS_ERR = 0;
constexpr size_t WS_TOKEN = 64;
constexpr size_t WS_BAR_ARRIVE = 256;  // own cache lines: polled by every workgroup
constexpr size_t WS_BAR_GEN = 384;
constexpr size_t WS_SEL_HINT = 512;     // per layer: the last k-th score key and a window half-width
constexpr size_t WS_CTRL_BYTES = 4096;
constexpr int WS_SEL_HINT_LAYERS = (int)((WS_CTRL_BYTES - WS_SEL_HINT) / 8);
constexpr int MLP_MAX_WG = 1024;  // partial rows the workspace holds (workgroups of one call)

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
inline size_t ws_z_offset() { return WS_CTRL_BYTES; }
inline size_t ws_partials_offset(const np_shape& s) {
  return align256(ws_z_offset() + (size_t)s.layers * s.rank * 4);
}
inline size_t ws_total(const np_shape& s) {
  // partial rows of d rounded up to whole 16-column blocks
  return align256(ws_partials_offset(s) + (size_t)MLP_MAX_WG * ((s.d_model + 15) / 16 * 16) * 4);
}

// Scratch of the allocation-free sparse MLP: NOALLOC_MAX_WG partial rows of
// at most NOALLOC_MAX_D fp32 columns (8 MiB per device).
constexpr int NOALLOC_MAX_WG = 256;
constexpr int NOALLOC_MAX_D = 8192;
constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)NOALLOC_MAX_WG * NOALLOC_MAX_D * 4;

inline int dtype_size(int dt) { return dt == NP_F32 ? 4 : 2; }
// elements per 16-byte vector
inline int vec_elems(int dt) { return 16 / dtype_size(dt); }

// ---------------------------------------------------------------------------
// launchers (defined in the .hip files; return hipError_t of the launch)
// ---------------------------------------------------------------------------
hipError_t launch_fill_state(const np_shape& s, const np_state& st, void* ws, hipStream_t stream);
hipError_t launch_predict(const np_shape& s, const void* h, const void* A, const void* B,
                          float* scores, void* ws, hipStream_t stream);
hipError_t launch_select(const np_shape& s, const float* scores, uint32_t* mask,
                         int32_t* active_ids, void* ws, hipStream_t stream);
// active_counts: nullptr for k active neurons per layer, else device [L'].
hipError_t launch_delta(const np_shape& s, int32_t token, const int32_t* active_ids,
                        const np_state& st, const np_delta_out& out, void* ws,
                        hipStream_t stream, const int32_t* active_counts = nullptr);
hipError_t launch_select_delta(const np_shape& s, int32_t token, const float* scores,
                               uint32_t* mask, int32_t* active_ids, const np_state& st,
                               const np_delta_out& out, void* ws, hipStream_t stream);
hipError_t launch_centroid_logits(const np_shape& s, const np_centroid_model& m,
                                  const void* feat, float* logits, hipStream_t stream);
hipError_t launch_centroid_active(const np_shape& s, const np_centroid_model& m,
                                  const float* logits, int32_t* centroid_ids, uint32_t* mask,
                                  int32_t* active_ids, int32_t* active_counts, void* ws,
                                  hipStream_t stream);
// host_storage: the storage is pinned host memory read over the host link
hipError_t launch_stage_gather(const np_shape& s, const np_delta_out& out, int layer_begin,
                               int layer_end, const void* storage, void* resident, void* ws,
                               hipStream_t stream, bool host_storage = false);
hipError_t launch_stage_scatter(const np_shape& s, const void* landing, const int32_t* rows,
                                int n_records, void* resident, hipStream_t stream);
hipError_t launch_dense_mlp(const np_shape& s, const void* weights, const void* x, void* y,
                            void* ws, hipStream_t stream);
// n_dev: nullptr for n_active rows, else the row count is n_dev[layer]
// (device), at most n_active.  thr: nullptr, or the eq. 1 threshold of each
// layer (device fp32 [L']).
// ids/slot_map: with active_slots == nullptr, row j is slot slot_map[ids[j]]
// (the layer's active ids and its row of the slot map).
hipError_t launch_sparse_mlp(const np_shape& s, int layer, const void* x, const void* resident,
                             const int32_t* active_slots, int n_active, void* y, void* ws,
                             hipStream_t stream, const int32_t* n_dev = nullptr,
                             const float* thr = nullptr, const int32_t* ids = nullptr,
                             const int32_t* slot_map = nullptr);
// np_sparse_mlp with its partial sums in the library's own device array
// (no workspace); device errors are OR-ed into *dev_error.
hipError_t launch_sparse_mlp_noalloc(const np_shape& s, int layer, const void* x,
                                     const void* resident, const int32_t* active_slots,
                                     int n_active, void* y, int32_t* dev_error,
                                     hipStream_t stream);
// activations of one layer over n tokens (matrix cores), acts [n][F] fp32
hipError_t launch_act_batch(const np_shape& s, const void* weights, const void* x, int n,
                            float* acts, hipStream_t stream);
// per row: the m-th smallest magnitude of n values (1 <= m <= n)
size_t percentile_ws_bytes(int rows);
hipError_t launch_percentile(const float* values, int rows, int64_t n, int64_t m, float* out,
                             void* ws, size_t ws_bytes, hipStream_t stream);
// eq. 1 masks and ascending ids of rows x F activations
hipError_t launch_threshold_active(const np_shape& s, const float* acts, int rows,
                                   const float* thr, uint32_t* mask, int32_t* active_ids,
                                   int32_t* active_counts, void* ws, hipStream_t stream);

// storage-tier file reads (np_file.cpp): io_uring, up to IO_QD_MAX requests
// in flight, runs cut into pieces of IO_PIECE bytes; an O_DIRECT file needs
// offsets, sizes and buffers aligned to IO_ALIGN bytes
constexpr int IO_QD_MAX = 256;
constexpr size_t IO_PIECE = (size_t)1 << 20;
constexpr int IO_ALIGN = 512;
struct ReadRun {
  char* dst;
  uint64_t offset;  // file offset
  size_t bytes;
};
int io_depth();  // NP_IO_QD clamped to [1, IO_QD_MAX], default IO_QD_MAX
bool file_is_direct(int fd);
// done (optional): called on the calling thread for each piece once it is
// read in full (dst, bytes), while the other reads are still in flight
typedef void (*PieceDone)(void* ctx, char* dst, size_t bytes);
np_status read_runs(int fd, const std::vector<ReadRun>& runs, int qd, PieceDone done = nullptr,
                    void* ctx = nullptr);

// host-side helpers shared by the ABI files (np_abi.cpp)
np_status fail(np_status st, const char* fmt, ...);
// Resident buffers whose staging failed after np_delta had already moved the
// slot map: the map names records that never arrived.  Every later staging
// or MLP call on such a buffer fails with NP_ERR_STATE until np_state_reset
// is given that buffer, which clears its mark (and no other).
void mark_resident_incomplete(const void* resident);
np_status check_resident(const char* fn, const void* resident);
void clear_incomplete_resident(const void* resident);
np_status hip_fail(hipError_t e, const char* what);
bool aligned16(const void* p);
np_status check_shape(const np_shape* s);

}  // namespace np
