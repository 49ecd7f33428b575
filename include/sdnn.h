/*
 * sdnn.h -- C ABI of the MI355X Sparse DNN inference library (libsdnn.so).
 *
 * Computes the Sparse DNN Challenge inference of Kepner et al. (2019):
 *   Sec. II, batched inference equation:  Y_{l+1} = h(Y_l W_l + B_l), with h(y) = min(YMAX, max(y, 0))
 *   (ReLU with the challenge's upper limit, Sec. II; YMAX = 32 in the Sec. V listing), the bias added
 *   only where Y_l W_l is nonzero (the Sec. V serial loop), for every layer l = 0..L-1;
 *   then the categories: the rows of the final Y with any entry > 0 (Sec. V, second timed step).
 *
 * Numerics: fp32. Every output is z = fma(y_{k_m}, w_m, ... fma(y_{k_0}, w_0, +0)) over the sources of
 * its column in ascending source order, one rounding per term; then t = z + b (one fp32 add) and
 * y = (z != 0) ? min(ymax, max(0, t)) : 0, with zeros written as +0. Results are therefore identical
 * on every run and match a sequential fp32 evaluation in that order bit for bit.
 *
 * Call order (Sec. V: download, load, set bias untimed; evaluate all layers and identify categories
 * timed; compare untimed):
 *   sdnn_create -> sdnn_load_layers (any chunks covering layers 0..L-1) -> [sdnn_infer ->
 *   sdnn_categories]* -> diagnostics -> sdnn_destroy.
 * The timed region of the challenge is sdnn_infer + sdnn_categories.
 *
 * Ownership: the library owns the handle and its device copies of the weights and biases. The caller
 * owns the input activations, the workspace, the stream and every host array; host arrays may be
 * reused as soon as a call returns. No call after sdnn_load_layers allocates device memory.
 *
 * Errors: no exception crosses the ABI. Every call returns an sdnn_status; sdnn_last_error() gives a
 * thread-local message for the last failure. SDNN_EINVAL, SDNN_ESTATE and SDNN_ERANGE leave the
 * handle unchanged. SDNN_EDEVICE (a HIP call failed) poisons the handle: every later call except
 * sdnn_destroy returns SDNN_EDEVICE.
 *
 * A handle is not thread-safe; use one handle per thread.
 */
#ifndef SDNN_H
#define SDNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sdnn_net sdnn_net;

typedef enum {
  SDNN_OK = 0,
  SDNN_EINVAL = 1,  /* an argument is malformed or out of range */
  SDNN_ENOMEM = 2,  /* a device or host allocation failed (only sdnn_create / sdnn_load_layers) */
  SDNN_EDEVICE = 3, /* a HIP call failed; the handle is poisoned */
  SDNN_ESTATE = 4,  /* call out of order (e.g. infer before every layer is loaded) */
  SDNN_ERANGE = 5   /* output capacity too small; the needed size is reported */
} sdnn_status;

/* Create a network of n_layers layers of n_neurons neurons each (Sec. II: N neurons per layer,
 * L layers). ymax is the upper limit of h (Sec. II; 32 in the challenge) and must be finite and > 0.
 * 1 <= n_neurons <= 65536, 1 <= n_layers <= 1000000. Host-only: touches no device. */
sdnn_status sdnn_create(sdnn_net **out, int32_t n_neurons, int32_t n_layers, float ymax);

/* Opt in (enable = 1) to kernels that exploit layers whose weights are all equal and whose biases
 * are all equal: such a layer is read as one weight, one bias and 16-bit source lists; layer 0 on
 * binary inputs is computed from counts of active sources; columns that share their source list are
 * computed once. Results are bit-identical to the default. Off by default, because the paper's
 * Sec. V lists exploiting the repetitive structure of weight and bias values among the things a
 * challenge submission should avoid: by default every layer reads each edge's weight and each
 * neuron's bias from memory. Host-only. Must precede the first sdnn_load_layers (SDNN_ESTATE
 * afterwards); enable other than 0 or 1 is SDNN_EINVAL. */
sdnn_status sdnn_enable_equal_value_kernels(sdnn_net *net, int32_t enable);

/* Load layers [l0, l0 + nl) (Sec. V: load the DNN; create the bias vectors b_l).
 * Weights in CSC, one column per output neuron j (Sec. II: W(i, j) != 0 connects neuron i to
 * neuron j, and rows y multiply W from the left, so column j lists the inputs of neuron j):
 *   col_ptr: nl * (n_neurons + 1) int64, host. Layer i's column j holds entries
 *            [col_ptr[i*(N+1) + j], col_ptr[i*(N+1) + j + 1]) of row_idx/val. Offsets are absolute
 *            indexes into row_idx/val, non-decreasing within a layer; layer i starts where layer i-1
 *            ends (col_ptr[i*(N+1)] == col_ptr[(i-1)*(N+1) + N]); col_ptr[0] may be nonzero.
 *   row_idx: int32 source neurons, in [0, N), strictly ascending within each column, host.
 *   val:     fp32 weights, finite, host.
 *   bias:    nl * n_neurons fp32, finite, host; bias[i*N + j] = b_l(j) for l = l0 + i.
 * A column may hold at most 4096 sources. Each layer may be loaded once. The call copies the data
 * into device memory it owns (allocated here, on the current device) and packs it into the layout
 * the kernels read; it synchronizes `hip_stream` (a hipStream_t, or NULL for the default stream)
 * before returning. With sdnn_enable_equal_value_kernels on, columns of a one-weight layer with 32
 * sources that share their source list (and so their output) are computed once when the next layer
 * is loaded right after it, in the same call or the next one; loading layers in ascending order
 * therefore never costs speed, and any order gives the same results. The first call on a handle
 * also creates the host-side objects the timed calls use (read-back events, pinned host words), so
 * that sdnn_infer and sdnn_categories allocate nothing. */
sdnn_status sdnn_load_layers(sdnn_net *net, int32_t l0, int32_t nl, const int64_t *col_ptr,
                             const int32_t *row_idx, const float *val, const float *bias,
                             void *hip_stream);

/* Bytes of device workspace sdnn_infer needs for n_rows input rows (activation buffers, live-row
 * lists, flags, counters). n_rows >= 0. Returns 0 for a NULL handle or negative n_rows. */
size_t sdnn_workspace_bytes(const sdnn_net *net, int64_t n_rows);

/* TIMED. Evaluate all layers (Sec. II batched equation) for the n_rows input rows in y0.
 *   y0:        device pointer, n_rows x n_neurons fp32, row-major (Sec. IV: one flattened input per
 *              row), finite; read-only, so the same y0 can be run again. Not needed after the call's
 *              work completes on the stream.
 *   workspace: device pointer, >= sdnn_workspace_bytes(net, n_rows) bytes, 256-byte aligned; owned
 *              by the caller, overwritten, must stay untouched until sdnn_categories returns and
 *              while diagnostics are read.
 *   hip_stream: hipStream_t (NULL = default stream) on which all work is enqueued.
 * Rows that become all zero are dropped from later layers: their activations stay zero for every W
 * and b, since Z = 0 gets no bias. The call enqueues layers in chunks and reads the live-row count
 * back from the device every few layers, so it may block until earlier layers finish; once no row
 * is live it stops enqueuing. Requires every layer to be loaded (SDNN_ESTATE otherwise). */
sdnn_status sdnn_infer(sdnn_net *net, const float *y0, int64_t n_rows, void *workspace,
                       size_t workspace_bytes, void *hip_stream);

/* TIMED. sdnn_infer for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same computation and results,
 * with the workspace taken from a 64 MiB array in the library's device memory instead of a caller
 * buffer. Allocates nothing (no hipMalloc, hipFree or allocating library call). The array is one per
 * device, shared by every handle and call on that device, and keeps the last call's contents: calls
 * that overlap on one device race, so serialize them (one stream, or wait for sdnn_categories) and
 * read a run's diagnostics (sdnn_live_counts, sdnn_final_rows) before the next static run on that
 * device. n_rows must satisfy sdnn_workspace_bytes(net, n_rows) <= 64 MiB; larger batches return
 * SDNN_ERANGE (nothing is enqueued). Other arguments and errors as for sdnn_infer. */
sdnn_status sdnn_infer_static(sdnn_net *net, const float *y0, int64_t n_rows, void *hip_stream);

/* TIMED. Wait for the last sdnn_infer and report its categories (Sec. V: the rows of the final
 * matrix with entries > 0): 0-based row indexes into y0, ascending, written to ids (host,
 * capacity entries). *count receives the number of categories. ids == NULL or capacity < count
 * returns SDNN_ERANGE with *count set (query mode). SDNN_ESTATE before any sdnn_infer. */
sdnn_status sdnn_categories(sdnn_net *net, int64_t *ids, int64_t capacity, int64_t *count);

/* Diagnostics (untimed). Live-row counts of the last sdnn_infer: counts[0] = input rows with any
 * nonzero entry, counts[l] = rows with any entry > 0 after layer l-1, for l = 1..n_layers (zeros
 * after the layer where no row was left). counts: host, n_layers + 1 entries. */
sdnn_status sdnn_live_counts(sdnn_net *net, int64_t *counts);

/* Diagnostics (untimed). Final activations of rows ids[0..n) (0-based, < n_rows of the last
 * sdnn_infer) into out_host (n x n_neurons fp32, row-major); rows that are not categories are all
 * zero. SDNN_EINVAL for an id out of range. */
sdnn_status sdnn_final_rows(sdnn_net *net, const int64_t *ids, int64_t n, float *out_host);

/* Diagnostics. enable == 1: every later sdnn_infer records a HIP event pair on its stream around
 * each layer's kernels (the layer SpMM with its fused epilogue; not the compaction), and
 * sdnn_categories adds the elapsed times to per-layer totals. enable == 2: the same for large
 * layers only (layers whose live rows take more than one round of tiles, or, for widths staged in
 * LDS, while more than 256 rows may be live), so that the event records do not slow the long tail
 * of layers with few rows. enable == 0 stops recording; other values are SDNN_EINVAL.
 * Creates its events here (needs the device); enabling again resets the totals. */
sdnn_status sdnn_set_profiling(sdnn_net *net, int32_t enable);

/* Diagnostics. Per-layer totals since profiling was enabled: ms[l] milliseconds over runs[l] timed
 * runs of layer l (0 for layers not recorded). ms, runs: host arrays of n_layers entries. */
sdnn_status sdnn_layer_times(sdnn_net *net, double *ms, int64_t *runs);

/* Kernel families reported by sdnn_layer_info. */
typedef enum {
  SDNN_KERNEL_NONE = 0,                 /* layer not run (every row had died) */
  SDNN_KERNEL_LDS_TILE = 1,             /* activation tiles staged in LDS (k_layer_lds) */
  SDNN_KERNEL_GLOBAL_TILE = 2,          /* fp32 feature-major tiles in global memory (k_layer_gfm) */
  SDNN_KERNEL_GLOBAL_TILE_CODES = 3,    /* one-byte dictionary codes of the inputs (k_layer_gfm_u8) */
  SDNN_KERNEL_GLOBAL_TILE_FEW_ROWS = 4, /* at most 8 tiles, whole chains in flight (k_layer_gfm_small) */
  SDNN_KERNEL_BITS = 5,                 /* layer 0 from bit-packed binary inputs (k_pack_bits, k_layer_bits) */
  SDNN_KERNEL_BITS_TO_CODES = 6,        /* the same, writing one-byte dictionary codes */
  SDNN_KERNEL_BITS_COUNT = 7,           /* layer 0 of a uniform layer on binary inputs, by bit-sliced counts
                                           (k_pack_bits, k_count_dict, k_layer_count); only with
                                           sdnn_enable_equal_value_kernels */
  SDNN_KERNEL_LDS_FUSED = 8,            /* every layer from this one on, in one launch that keeps each
                                           workgroup's rows in LDS (k_layers_lds); the launch is counted
                                           at its first layer, later layers report 0 launches */
  SDNN_KERNEL_GLOBAL_TILE_CODES16 = 9   /* two-byte dictionary codes of the inputs, for inputs of 257 to
                                           4096 distinct values (k_layer_gfm_u8 on 16-bit codes) */
} sdnn_kernel_kind;

/* Diagnostics (untimed). For each layer of the last sdnn_infer: the kernel family that ran it
 * (sdnn_kernel_kind) and its number of kernel launches, those that encoded its inputs included (for
 * layers timed with events, the event pair spans these launches). kernel, launches: host arrays of
 * n_layers entries. */
sdnn_status sdnn_layer_info(sdnn_net *net, int32_t *kernel, int32_t *launches);

/* Free the handle and its device memory. NULL is a no-op. */
void sdnn_destroy(sdnn_net *net);

/* Thread-local description of the last failed call ("" if none). */
const char *sdnn_last_error(void);

/* Which kernel family the handle uses for its width: 0 = activation tiles staged in LDS,
 * 1 = tiles gathered from global memory (widths too large for LDS). -1 for NULL. */
int32_t sdnn_kernel_path(const sdnn_net *net);

#ifdef __cplusplus
}
#endif

#endif /* SDNN_H */
