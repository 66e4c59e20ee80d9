/*
 * neuroprefetch.h -- C ABI of the per-token decode hot path of NeuroPrefetcher
 * ("Storage-Aware Sparse LLM Inference via Delta Prefetching", arXiv 2608.22643),
 * built for one AMD Instinct MI355X (gfx950).
 *
 * One decode token runs five steps (paper Sec. 3.1, "System Overview"; Sec. 3.4,
 * "Predictive Delta Prefetching"; Sec. 3.5, "I/O Path"):
 *
 *   np_predict     score the MLP neurons of every downstream layer in one pass
 *   np_select      top-k of the scores -> one fixed-size active set per layer
 *   np_delta       active set vs. the GPU-resident row buffer -> incoming rows,
 *                  evicted slots, hits; updates the slot map (Sec. 3.4, eqs. 2-3)
 *                  (np_select_delta: both in one call)
 *   np_stage_rows  incoming neuron records, storage tier -> their device slots
 *                  (np_stage_file: the storage tier in a file, read with io_uring)
 *   np_sparse_mlp  ReLU-gated MLP over the resident active rows of one layer
 *
 * and, for the paper's own predictor (centroid IDs, variable-size sets):
 *
 *   np_centroid_select  centroid heads -> gate/up centroid ids -> the
 *                       intersected active set of every layer (Sec. 3.3-3.4)
 *   np_delta_n, np_sparse_mlp_n   np_delta / np_sparse_mlp with per-layer
 *                       active counts read on the device
 *
 * and np_dense_mlp for the layers of a dense prefix (Sec. 3.1).
 *
 * The MLP calls evaluate either gated form (np_shape.act): the ReLU-gated
 * MLP of the synthetic models or the SwiGLU MLP of the paper's evaluated
 * models (Sec. 4).  For the magnitude-threshold sparsity of Sec. 3.2 (eq. 1):
 *
 *   np_sparse_mlp_t      np_sparse_mlp with eq. 1 applied to each active row
 *   np_act_batch         activations of one layer over a batch of tokens
 *                        (matrix cores; the calibration input)
 *   np_percentile        per-layer alpha-th percentile of |activation|: T(l, alpha)
 *   np_threshold_active  eq. 1 as an active set: |a| >= T -> mask + ascending ids
 *
 * Conventions shared by every call
 * --------------------------------
 *  - extern "C"; plain pointers and sizes only.  All memory is owned by the
 *    caller; no call allocates or frees device or host memory
 *    (np_sparse_mlp_noalloc's scratch is a device array of the library
 *    itself, 8 MiB per device, present once the library's code is loaded on
 *    that device).  The staging path keeps a few HIP events per pinned
 *    staging buffer it is given and one pool of packing threads per process,
 *    created on first use (see np_stage_rows), and the file tier one io_uring
 *    ring of 256 entries per process (see np_stage_file).
 *  - "device" pointers point into memory of the current HIP device.  Device
 *    pointers must be 16-byte aligned.  Every call is asynchronous on the HIP
 *    stream it is given (0 = the null stream) unless stated otherwise.
 *  - Host-side argument validation runs first; when it fails nothing is
 *    enqueued and the call returns NP_ERR_INVALID_ARG or NP_ERR_CAPACITY.
 *    np_last_error() then gives a detail string (thread-local).
 *  - A failing HIP runtime call returns NP_ERR_HIP.  Data errors that only the
 *    device can see (a NaN score, an active row that is not resident, a slot
 *    map that disagrees with its inverse) set bits in a sticky error word in
 *    the device workspace; read it with np_device_error().
 *  - Calls that share a workspace or a state must not run concurrently.
 *
 * Shapes and layouts (np_shape)
 * -----------------------------
 *  L' = layers (downstream layers, i.e. layers 1..N-1 of an N-layer model),
 *  d  = d_model, F = d_ffn (MLP intermediate size), r = predictor rank,
 *  k  = active rows per layer, C = resident slots per layer.
 *  w  = wdtype (MLP records and predictor factors), a = adtype (h, x, y).
 *  act = gated activation of the MLP neurons (np_act).
 *  Requirements: wdtype == adtype; 1 <= k <= C <= F <= 65535; k <= 8192;
 *  L' >= 1; d and r multiples of 8 for 16-bit types and of 4 for fp32;
 *  d <= 16384 (16-bit) or 8192 (fp32); r <= 1024 (16-bit) or 512 (fp32);
 *  C * 3d * sizeof(w) < 2^31 (one layer's resident buffer below 2 GiB).
 *  k > C is NP_ERR_CAPACITY; any other violation NP_ERR_INVALID_ARG.
 *
 *  Neuron record (Sec. 3.5, neuron-centric layout): row n of gate, row n of up
 *  and row n of down^T (down transposed offline so all three share one shape),
 *  3*d elements of type w, contiguous, no padding.  Storage tier:
 *  [L'][F][3d] (record n of layer l at ((l*F)+n)*3d).  Device resident
 *  buffer: [L'][C][3d] (slot s of layer l at ((l*C)+s)*3d).
 */
#ifndef NEUROPREFETCH_H
#define NEUROPREFETCH_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum np_status {
  NP_OK = 0,
  NP_ERR_INVALID_ARG = 1, /* null/misaligned pointer, bad size or dtype */
  NP_ERR_CAPACITY = 2,    /* k > C, staging buffer smaller than one record, ... */
  NP_ERR_HIP = 3,         /* a HIP runtime call failed; detail in np_last_error() */
  NP_ERR_UNSUPPORTED = 4, /* valid request this library does not implement */
  NP_ERR_STATE = 5,       /* a staging into this resident buffer failed part-way: calls on it
                             fail until np_state_reset */
  NP_ERR_IO = 6           /* a storage-tier file read failed (detail in np_last_error()) */
} np_status;

typedef enum np_dtype { NP_F32 = 0, NP_F16 = 1, NP_BF16 = 2 } np_dtype;

/* Gated activation of an MLP neuron with gate sum g and up sum u:
 * NP_ACT_RELU a = max(g, 0) * u; NP_ACT_SWIGLU a = SiLU(g) * u with
 * SiLU(g) = g / (1 + exp(-g)) (the SwiGLU MLP of the paper's models, Sec. 4;
 * exp is HIP's expf, the division IEEE fp32). */
typedef enum np_act { NP_ACT_RELU = 0, NP_ACT_SWIGLU = 1 } np_act;

/* Device error word bits (sticky, OR-ed; see np_device_error). */
#define NP_DEVERR_NAN_SCORE    0x1  /* a NaN score, logit or activation was read */
#define NP_DEVERR_NOT_RESIDENT 0x2  /* a slot outside [0, C) or id outside [0, F) */
#define NP_DEVERR_STATE        0x4  /* inconsistent state or plan (ids, slots, counts) */
#define NP_DEVERR_SPIN_LIMIT   0x8  /* a bounded in-kernel wait gave up */
#define NP_DEVERR_OVERFLOW     0x10 /* an active set larger than k was cut to k */

typedef struct np_shape {
  int32_t layers;   /* L' */
  int32_t d_model;  /* d */
  int32_t d_ffn;    /* F */
  int32_t rank;     /* r */
  int32_t k;        /* active rows per layer */
  int32_t capacity; /* C: resident slots per layer */
  int32_t wdtype;   /* np_dtype of MLP records and predictor factors */
  int32_t adtype;   /* np_dtype of activations h, x, y */
  int32_t act;      /* np_act of the MLP neurons */
} np_shape;

/* Residency state of every downstream layer, device memory, int32.
 * slot_of   [L'][F]: the slot map S of Sec. 3.4; slot of neuron n or -1.
 * neuron_of [L'][C]: inverse map; neuron held by slot s or -1.
 * last_used [L'][F]: last token at which neuron n was active, -1 if never
 *                    (drives least-recently-used eviction when C > k). */
typedef struct np_state {
  int32_t* slot_of;
  int32_t* neuron_of;
  int32_t* last_used;
} np_state;

/* Outputs of np_delta, device memory.  Each list is [L'][k] int32 (row l
 * holds layer l's list; only the first counts[l][.] entries are defined).
 * counts [L'][4] = { n_in, n_hit, n_ev, n_free_used = n_in - n_ev }. */
typedef struct np_delta_out {
  int32_t* in_ids;       /* incoming neurons, ascending */
  int32_t* in_slots;     /* slot given to in_ids[j], ascending */
  int32_t* ev_ids;       /* evicted neurons, ascending */
  int32_t* ev_slots;     /* the slot ev_ids[j] held before eviction */
  int32_t* hit_ids;      /* active neurons already resident, ascending */
  int32_t* active_slots; /* slot of active_ids[j] after the update, k per layer */
  int32_t* counts;
} np_delta_out;

/* The centroid-ID predictor (Sec. 3.3, third stage, and Sec. 3.4): 2 L'
 * linear heads over K centroids, gate heads of every downstream layer first,
 * then up heads, and a bank of sparse binary centroid masks per layer and
 * projection.  All device memory.
 * heads [2][L'][K][D] of type w (row c of head h: the logit weights of
 * centroid c); bank [2][L'][K][ceil(F/32)] uint32 (bit n%32 of word n/32 set
 * when centroid c keeps neuron n; pad bits ignored).  Requirements:
 * 1 <= K <= 4096; D a multiple of 8 (16-bit types) or 4 (fp32), D <= 16384
 * (16-bit) or 8192 (fp32). */
typedef struct np_centroid_model {
  int32_t n_centroids; /* K */
  int32_t feat_dim;    /* D */
  const void* heads;
  const uint32_t* bank;
} np_centroid_model;

/* Host copy of the parts of np_delta_out that staging needs ([L'][4] and
 * [L'][k] int32, any host memory; pinned makes the device->host copy async). */
typedef struct np_stage_plan {
  const int32_t* counts;
  const int32_t* in_ids;
  const int32_t* in_slots;
} np_stage_plan;

/* Text of a status code; never NULL. */
const char* np_status_str(int32_t status);

/* Detail of the last failing call on this thread ("" if none). */
const char* np_last_error(void);

/* Validates a shape (the requirements listed above).  Host only. */
np_status np_shape_check(const np_shape* shape);

/* Bytes of device workspace ("dev_ws") the calls below need for this shape
 * (one workspace serves all calls of one decode stream), and, in
 * *pinned_host_bytes (nullable), the pinned host memory one decode stream
 * uses to stage from a host or file tier: the plan copy (counts, in_ids,
 * in_slots: L' (4 + 2k) int32, rounded up to 4 KiB) plus the staging area
 * np_stage_rows is tuned for: four pieces of 16 MiB (at least one record and
 * its row index each, in 4 KiB pages).  Host only. */
np_status np_workspace_size(const np_shape* shape, size_t* dev_ws_bytes,
                            size_t* pinned_host_bytes);

/* Cold start (Sec. 3.1 last paragraph; Sec. 3.4 "the first token has no
 * previous active set"): sets every entry of slot_of, neuron_of and last_used
 * to -1 with a fill kernel on `stream`, and clears the device error word and
 * the workspace counters.  After it, np_delta on the next token gives every
 * active neuron a slot (slots 0..k-1 in ascending neuron order).
 * dev_resident (nullable): the resident buffer this state describes; its
 * NP_ERR_STATE mark is lifted.  A staging that fails at run time
 * (NP_ERR_HIP, NP_ERR_IO or NP_ERR_UNSUPPORTED from np_stage_rows,
 * np_stage_file or np_stage_gather) may have placed only part of a delta
 * whose slot map np_delta had already written, so that resident buffer is
 * marked and every later staging or sparse-MLP call on it returns
 * NP_ERR_STATE until the decode restarts from a cold start that names it.
 * Marks of other resident buffers are left alone.  Argument errors mark
 * nothing.  A mark is kept by the buffer's base address: a marked buffer
 * that is freed leaves its mark on the address, so a new buffer allocated
 * there is refused the same way until a reset names it. */
np_status np_state_reset(const np_shape* shape, const np_state* state,
                         const void* dev_resident, void* dev_ws, hipStream_t stream);

/* Activity predictor (Sec. 3.1 step 2, Sec. 3.3 role: one pass after layer 0
 * scores every downstream layer).  Low-rank form per downstream layer l:
 *     z_l = A_l h          (r values, fp32, kept in dev_ws)
 *     scores[l] = B_l z_l  (F values, fp32)
 * h [d] of type a; A [L'][r][d] and B [L'][F][r] of type w, row-major;
 * scores [L'][F] fp32; all device.  Two kernels on `stream`. */
np_status np_predict(const np_shape* shape, const void* h, const void* A,
                     const void* B, float* scores, void* dev_ws,
                     hipStream_t stream);

/* Fixed-size active sets (Sec. 3.4: every active set has the same size).
 * For each layer: the k neurons with the largest score; a tie at the k-th
 * score goes to the smaller neuron id; -0.0 equals +0.0; a NaN sets
 * NP_DEVERR_NAN_SCORE (its neuron is then treated as the smallest score).
 * scores [L'][F] fp32 device -> mask [L'][ceil(F/32)] uint32 (bit n%32 of
 * word n/32, LSB first, pad bits 0) and active_ids [L'][k] int32 ascending.
 * One workgroup per layer on `stream`. */
np_status np_select(const np_shape* shape, const float* scores, uint32_t* mask,
                    int32_t* active_ids, void* dev_ws, hipStream_t stream);

/* token argument of np_delta: use the workspace's step counter (below). */
#define NP_TOKEN_AUTO (-1)

/* Delta against the resident set (Sec. 3.4, eqs. 2-3 and the slot-map
 * paragraph), for token index `token` >= 0:
 *   hits H = active neurons with slot_of >= 0; incoming I = the rest;
 *   free slots Fr = slots with neuron_of == -1 (ascending);
 *   if |I| > |Fr|, the m = |I|-|Fr| victims are the resident, non-active
 *   neurons with the smallest (last_used, id); their slots join the pool;
 *   the pool (ascending) is paired with I (ascending); last_used := token for
 *   every active neuron.  With C == k this is exactly D_in = A_t \ A_{t-1},
 *   D_out = A_{t-1} \ A_t.
 * active_ids [L'][k] ascending (np_select output), device.  `state` is read
 * and updated in place; `out` lists are written.  One workgroup per layer.
 * token == NP_TOKEN_AUTO: the index is read on the device from a step counter
 * in dev_ws (np_state_reset sets it to 0), and a second kernel advances the
 * counter by one after the delta.  With it a decode step has no per-token
 * argument besides its input buffers, so a captured HIP graph of the step can
 * be replayed as is; tokens 0, 1, 2, ... then match explicit indices.
 * token < -1 is NP_ERR_INVALID_ARG. */
np_status np_delta(const np_shape* shape, int32_t token,
                   const int32_t* active_ids, const np_state* state,
                   const np_delta_out* out, void* dev_ws, hipStream_t stream);

/* np_select followed by np_delta (Sec. 3.4: the fixed-size active set and
 * its delta against the resident set) in one call: the same arguments as the
 * two calls, the same results bit for bit (mask, active_ids, the state and
 * every `out` list), the same error reporting (NP_DEVERR_NAN_SCORE,
 * NP_DEVERR_STATE).  Where the layer fits one workgroup's local memory
 * (F <= 16384, C <= 8192, k <= 4096) both steps run in one kernel per layer
 * that reads slot_of and neuron_of once into local memory at entry, together
 * with the scores; other shapes run np_select's and np_delta's kernels.  With
 * token == NP_TOKEN_AUTO a second kernel advances the step counter, as in
 * np_delta. */
np_status np_select_delta(const np_shape* shape, int32_t token, const float* scores,
                          uint32_t* mask, int32_t* active_ids, const np_state* state,
                          const np_delta_out* out, void* dev_ws, hipStream_t stream);

/* Staging through pinned host memory and hipMemcpyAsync (Sec. 3.5: incoming
 * ids sorted and coalesced into contiguous ranges, one token-level batch for
 * all layers, staging capacity-bounded with chunked submit-and-scatter).
 * For layers [layer_begin, layer_end):
 *   resident[l][in_slots[l][j]] <- storage[l][in_ids[l][j]],  j < counts[l][0].
 * plan: host copy of np_delta's counts/in_ids/in_slots (read synchronously).
 * host_storage: [L'][F][3d] records, pinned host memory (hipHostMalloc).
 * dev_resident: [L'][C][3d] device.
 * host_staging / staging_bytes (pinned host, 16-byte aligned): a ring of up
 * to 4 pieces (4 KiB multiples) into which the host packs records (8
 * threads), rec = 3d*sizeof(w) bytes each, followed by their int32
 * destination rows (layer * C + slot); a piece of n records is sent as one
 * block of n * (rec + 4) bytes with one hipMemcpyAsync on `side` into the
 * landing area, and one scatter kernel then moves its records into their
 * slots.
 * dev_landing / landing_bytes (device, 16-byte aligned): a ring of landed
 * blocks, each at a 16-byte boundary; it must hold one record and its row
 * (landing_bytes >= rec + 4); a piece holds at most what the whole ring
 * holds, and the ring wraps to its start when what is left of it cannot
 * hold the next piece.  The scatters run on a stream the library keeps per staging
 * buffer (default priority), each ordered after its block's copy by an
 * event, so the copies run back to back on the copy engine; copies into a
 * wrapped ring wait for the scatters before them.
 * wait_before (nullable): the scatters of this call wait on it (orders the
 * writes into dev_resident after the previous token's MLP reads).
 * layer_ready (nullable, [L'] events): at the end of a layer, once the
 * layers since the last recorded event hold 8 MiB of records
 * (NP_STAGE_GROUP_MIB), the open piece is sent, and events of those layers
 * are recorded after its scatter; event l thus follows the scatter that
 * places layer l's last record, and these events are the call's completion
 * signal.  Without layer_ready, `side` is made to
 * wait for the call's last scatter, so later work on `side` follows the whole
 * staging.  The host blocks only to reuse a staging piece whose copy has not
 * finished.  State kept between calls (pending copies,
 * the rings' positions, the scatter stream) is per staging buffer: calls
 * with different staging buffers are independent; calls with the same one
 * must come from one thread at a time.  On a failure after some pieces were
 * copied, those records are still scattered before the call returns the
 * error.  Returns NP_ERR_CAPACITY if the landing area or a staging piece
 * holds no record (with its row index). */
np_status np_stage_rows(const np_shape* shape, const np_stage_plan* plan,
                        int32_t layer_begin, int32_t layer_end,
                        const void* host_storage, void* dev_resident,
                        void* host_staging, size_t staging_bytes,
                        void* dev_landing, size_t landing_bytes,
                        hipStream_t side, hipEvent_t wait_before,
                        hipEvent_t* layer_ready);

/* np_stage_rows with the storage tier in a file (Sec. 3.5, I/O path): the
 * file holds the [L'][F][3d] records starting at byte file_offset (the
 * neuron-centric, layer-major layout).  The coalesced record ranges of each
 * staging piece are read through Linux io_uring with up to 256 reads in
 * flight (NP_IO_QD lowers it) into io_buffer, each finished read copied into
 * the pinned piece while the others are in flight, then sent and scattered
 * as in np_stage_rows.  io_buffer: ordinary host memory of io_buffer_bytes
 * (a piece holds at most io_buffer_bytes of records), owned by the caller;
 * NULL reads straight into the pinned pieces of host_staging.  Memory pinned through the HIP runtime cannot be the target
 * of a direct (O_DIRECT) read on this platform (the read fails with EFAULT),
 * so a direct-I/O descriptor needs io_buffer.  fd: a readable descriptor
 * owned by the caller; opened with O_DIRECT, the reads bypass the page cache
 * and the record size, file_offset and the read target must be multiples of
 * 512 bytes.  A failed or short read (end of file) returns NP_ERR_IO; the
 * pieces copied before it are still scattered.  Everything else as
 * np_stage_rows. */
np_status np_stage_file(const np_shape* shape, const np_stage_plan* plan,
                        int32_t layer_begin, int32_t layer_end, int32_t fd,
                        int64_t file_offset, void* dev_resident, void* host_staging,
                        size_t host_staging_bytes, void* io_buffer, size_t io_buffer_bytes,
                        void* dev_landing, size_t dev_landing_bytes, hipStream_t side,
                        hipEvent_t wait_before, hipEvent_t* layer_ready);

/* Host-side record gather from a storage-tier file (the reads of
 * np_stage_file without the device steps): dst[j] <- the record_bytes
 * record at file_offset + ids[j] * record_bytes, for j < n, with runs of
 * consecutive ids read as one range and up to 256 reads in flight through
 * io_uring.  dst: host memory of n * record_bytes bytes (ordinary memory
 * for an O_DIRECT fd, see np_stage_file).  With an O_DIRECT fd, file_offset,
 * record_bytes and dst must be multiples of 512.  Returns
 * NP_ERR_IO when a read fails or the file ends early.  Synchronous; calls
 * from several threads are serialised. */
np_status np_read_records(int32_t fd, int64_t file_offset, int64_t record_bytes,
                          const int32_t* ids, int32_t n, void* dst);

/* Staging without a host round trip: one kernel per call copies, for layers
 * [layer_begin, layer_end), resident[l][in_slots[l][j]] <- storage[l][in_ids[l][j]]
 * reading counts/in_ids/in_slots straight from np_delta's device output.
 * `storage` is [L'][F][3d] in device memory (a storage tier kept in HBM) or in
 * pinned host memory mapped into the device address space (the kernel then
 * reads it over the host link, as the paper's mapped staging does, Sec. 3.5).
 * An id or slot outside [0, F) x [0, C) sets NP_DEVERR_NOT_RESIDENT in
 * dev_ws and that record is skipped.  Asynchronous on `stream`; no host
 * synchronisation. */
np_status np_stage_gather(const np_shape* shape, const np_delta_out* out,
                          int32_t layer_begin, int32_t layer_end,
                          const void* storage, void* dev_resident,
                          void* dev_ws, hipStream_t stream);

/* Sparse MLP of one downstream layer over its resident active rows
 * (Sec. 3.4: the slot map locates each active row; row order is irrelevant;
 * Sec. 3.3: the down projection's output stays dense):
 *     g_j = gate_j . x,  u_j = up_j . x,  y = sum_j act(g_j, u_j) * downT_j
 * with act the gated form shape->act (max(g, 0) * u or SiLU(g) * u)
 * where row j is slot active_slots[j] (j < n_active) of layer `layer` of
 * dev_resident.  x [d] and y [d] of type a, device; accumulation in fp32 and
 * one rounding of y to type a.  A slot outside [0, C) sets
 * NP_DEVERR_NOT_RESIDENT and is skipped.  Two kernels on `stream` (rows into
 * per-workgroup fp32 partials in dev_ws, then a column reduction in a fixed
 * order: deterministic); call it once per layer, in layer order.
 * n_active = 0 gives y = 0.
 * With the environment variable NP_MLP_FUSED=1 the reduction runs inside the
 * rows kernel after a grid-wide barrier (one kernel) when the whole grid fits
 * on the device at once (an occupancy query at launch).  The barrier needs
 * every workgroup of the grid resident together, so nothing else may hold
 * compute units while it runs: no other np_sparse_mlp on the device, no
 * staging kernel on another stream (np_stage_gather or np_stage_rows'
 * scatter of an overlapped step), no kernel of the caller's.  Its wait is
 * bounded and sets NP_DEVERR_SPIN_LIMIT (y then undefined until
 * np_state_reset) if the grid never meets.  The default two-kernel path has
 * no such condition.  NP_MLP_COLSPLIT=1 selects a single kernel without partial
 * sums (16-bit records, d a multiple of 512, at most 4 * d / 8 rows; each
 * workgroup owns 16 columns of y) under the same barrier and conditions.
 * dev_ws must have been zeroed or passed to np_state_reset before its first
 * use. */
np_status np_sparse_mlp(const np_shape* shape, int32_t layer, const void* x,
                        const void* dev_resident, const int32_t* active_slots,
                        int32_t n_active, void* y, void* dev_ws,
                        hipStream_t stream);

/* np_sparse_mlp for callers that cannot allocate device memory or hand over
 * a workspace (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same computation, kernels, launch shape and
 * summation order as np_sparse_mlp, so y is bit-identical to np_sparse_mlp's
 * for the same inputs.  The per-workgroup partial sums live in the library's
 * own device array of 8 MiB per device (at most 256 workgroups of d <= 8192
 * fp32 columns), held from the first call on a device until the process ends;
 * the call itself allocates nothing.  dev_error: device int32 (4-byte
 * aligned) into which the kernels OR NP_DEVERR_* bits (the caller clears and
 * reads it).  d_model > 8192 returns NP_ERR_CAPACITY; the opt-in
 * single-kernel paths (NP_MLP_FUSED, NP_MLP_COLSPLIT) are never taken.  All
 * calls on one device share that array: calls that overlap in time on one
 * device (two streams, two threads) race and give undefined y.  Everything
 * else as np_sparse_mlp. */
np_status np_sparse_mlp_noalloc(const np_shape* shape, int32_t layer, const void* x,
                                const void* dev_resident, const int32_t* active_slots,
                                int32_t n_active, void* y, int32_t* dev_error,
                                hipStream_t stream);

/* np_sparse_mlp in the form of the paper's statement (Sec. 3.4: the slot map
 * locates each active row): row j is slot slot_of[active_ids[j]] of layer
 * `layer`.  active_ids: the layer's n_active active neuron ids (np_select's
 * row for the layer); slot_of: the layer's row of the slot map
 * (state.slot_of + layer * F), both device int32 with 4-byte alignment.  An
 * id outside [0, F) or a slot outside [0, C) sets NP_DEVERR_NOT_RESIDENT and
 * the row is skipped.  The kernels look the slot up themselves (one more
 * dependent load than np_sparse_mlp, which takes np_delta's active_slots,
 * the same lookup already applied); for the same rows in the same order both
 * give the same bits.  Everything else as np_sparse_mlp. */
np_status np_sparse_mlp_ids(const np_shape* shape, int32_t layer, const void* x,
                            const void* dev_resident, const int32_t* active_ids,
                            const int32_t* slot_of, int32_t n_active, void* y, void* dev_ws,
                            hipStream_t stream);

/* Centroid-ID prediction and the intersected active sets (Sec. 3.3: each
 * head selects its highest-scoring centroid; Sec. 3.4: the active set of a
 * layer is the intersection of its gate and up centroid masks):
 *   logits[h][c] = heads[h][c] . feat            (fp32, [2][L'][K])
 *   centroid_ids[h] = argmax_c logits[h][c]      (ties: the smaller c; [2][L'])
 *   mask[l] = bank[0][l][gate id] & bank[1][l][up id]   ([L'][ceil(F/32)])
 *   active_ids[l] = members of mask[l] ascending ([L'][k]), active_counts[l]
 * feat [D] of type a.  Lists hold at most k ids (the buffer capacity of a
 * layer): a larger intersection keeps its k smallest ids (mask keeps every
 * member) and sets NP_DEVERR_OVERFLOW; a NaN logit sets NP_DEVERR_NAN_SCORE
 * and never wins.  Entries of active_ids past the count are not written.
 * Two kernels on `stream`. */
np_status np_centroid_select(const np_shape* shape, const np_centroid_model* model,
                             const void* feat, float* logits, int32_t* centroid_ids,
                             uint32_t* mask, int32_t* active_ids,
                             int32_t* active_counts, void* dev_ws,
                             hipStream_t stream);

/* np_delta for active sets of variable size: layer l has active_counts[l]
 * (device int32, 0..k) neurons, active_ids[l][0..count) ascending.  Every
 * output and the state update follow np_delta with k replaced by the count;
 * active_slots[l] is written for the first count entries only.  A count
 * outside [0, k] sets NP_DEVERR_STATE and is clamped. */
np_status np_delta_n(const np_shape* shape, int32_t token,
                     const int32_t* active_ids, const int32_t* active_counts,
                     const np_state* state, const np_delta_out* out,
                     void* dev_ws, hipStream_t stream);

/* np_sparse_mlp over the first active_counts[layer] entries of active_slots
 * (active_counts: device int32 [L'], read on the device, so a count produced
 * on the GPU needs no host round trip; active_slots and active_counts need
 * 4-byte alignment only, so a layer's row of a [L'][k] list can be passed).
 * A count outside [0, k] sets NP_DEVERR_STATE and is clamped. */
np_status np_sparse_mlp_n(const np_shape* shape, int32_t layer, const void* x,
                          const void* dev_resident, const int32_t* active_slots,
                          const int32_t* active_counts, void* y, void* dev_ws,
                          hipStream_t stream);

/* Dense MLP of one layer of the dense prefix (Sec. 3.1: the first d layers
 * keep their MLP weights fully resident and run dense): the np_sparse_mlp
 * computation over all F neurons of `weights`, one layer's [F][3d] records of
 * type w in the storage layout (gate | up | down^T per neuron), device.
 * Requires F * 3d * sizeof(w) < 2^31.  x [d], y [d] of type a.  Two kernels on
 * `stream`. */
np_status np_dense_mlp(const np_shape* shape, const void* weights, const void* x, void* y,
                       void* dev_ws, hipStream_t stream);

/* np_sparse_mlp with the magnitude threshold of eq. 1 (Sec. 3.2) applied to
 * each active row: a_j = act(g_j, u_j) is replaced by 0 when
 * |a_j| < thresholds[layer] (fp32 comparison), so
 *     y = sum_j [|a_j| >= T] a_j downT_j.
 * thresholds: device fp32 [L'] (T of every downstream layer, e.g. from
 * np_percentile), or NULL for no threshold (T = 0 keeps every row too).
 * active_counts: NULL for n_active rows, else device int32 [L'] read on the
 * device as in np_sparse_mlp_n, with the row count min(count, n_active) and
 * a count outside [0, n_active] setting NP_DEVERR_STATE.  active_slots,
 * active_counts and thresholds need 4-byte alignment.  Everything else as
 * np_sparse_mlp (n_active in [0, C]). */
np_status np_sparse_mlp_t(const np_shape* shape, int32_t layer, const void* x,
                          const void* dev_resident, const int32_t* active_slots,
                          int32_t n_active, const int32_t* active_counts,
                          const float* thresholds, void* y, void* dev_ws,
                          hipStream_t stream);

/* Activations of one layer over a batch of tokens, the A(i, l) = f_l(x_i) that
 * Sec. 3.2 collects to set the per-layer thresholds:
 *     acts[i][f] = act(gate_f . x_i, up_f . x_i)     (i < n, f < F)
 * weights: one layer's [F][3d] records of type w (storage layout), device;
 * x: [n][d] of type a, device; acts: [n][F] fp32, device.  The two
 * projections are matrix products over the batch, run on the matrix cores
 * (MFMA, fp32 accumulation); acts is not rounded further.  Requires
 * 1 <= n <= 65536, F * 3d * sizeof(w) < 2^31 and n * d * sizeof(a) < 2^31.
 * A launch per 128 tokens on `stream`; dev_ws is not used (may be NULL). */
np_status np_act_batch(const np_shape* shape, const void* weights, const void* x, int32_t n,
                       float* acts, void* dev_ws, hipStream_t stream);

/* Per row r of `values` ([rows][n] fp32, device): the alpha-th percentile of
 * the magnitudes |values[r][.]|, the threshold T(l, alpha) of Sec. 3.2 when
 * row r holds layer l's calibration activations.  Nearest rank: out[r] is
 * the m-th smallest magnitude, m = ceil(alpha * n / 100) computed in double
 * on the host and clamped to [1, n], so out[r] is one of the magnitudes and
 * eq. 1 zeroes fewer than m of them.  alpha in [0, 100]; 1 <= rows <= 65535;
 * 1 <= n < 2^31; rows * n * 4 bytes of values.  out: device fp32 [rows].  A
 * NaN value sets NP_DEVERR_NAN_SCORE (out[r] is then undefined).  Radix
 * selection on the magnitude bits, three passes over each row.
 * dev_ws_bytes: the size of dev_ws (at least 64: the error word).  With at
 * least NP_PERCENTILE_WS_BYTES(rows) bytes, n > 32768 and rows < 1024, every
 * row is spread over several workgroups (per-row histograms and selection
 * state in dev_ws past its first 4096 bytes, which the call overwrites;
 * seven kernels on `stream`); otherwise one workgroup per row (one kernel)
 * and dev_ws holds only the error word.  Either way the result is the same. */
#define NP_PERCENTILE_WS_BYTES(rows) (4352 + 8208 * (size_t)(rows))
np_status np_percentile(const float* values, int32_t rows, int64_t n, double alpha, float* out,
                        void* dev_ws, size_t dev_ws_bytes, hipStream_t stream);

/* Eq. 1 as an active set, in np_select's layout: for each row r of acts
 * ([rows][F] fp32, device) with threshold thresholds[r] (device fp32
 * [rows]), neuron f is active when |acts[r][f]| >= thresholds[r].  mask:
 * [rows][ceil(F/32)] uint32 (bit f%32 of word f/32); active_ids: [rows][k]
 * ascending (only the first active_counts[r] entries are written);
 * active_counts: [rows] int32, all device.  A row with more than k active
 * neurons lists its k smallest ids, keeps every member in its mask, counts k
 * and sets NP_DEVERR_OVERFLOW; a NaN activation sets NP_DEVERR_NAN_SCORE.
 * F and k from `shape`; 1 <= rows <= 65535. */
np_status np_threshold_active(const np_shape* shape, const float* acts, int32_t rows,
                              const float* thresholds, uint32_t* mask, int32_t* active_ids,
                              int32_t* active_counts, void* dev_ws, hipStream_t stream);

/* Waits for `stream`, then returns the sticky device error word in *code
 * (0 = none; NP_DEVERR_* bits otherwise).  Synchronous. */
np_status np_device_error(const void* dev_ws, hipStream_t stream, int32_t* code);

#ifdef __cplusplus
}
#endif

#endif /* NEUROPREFETCH_H */
