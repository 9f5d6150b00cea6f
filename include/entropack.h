/*
 * entropack.h -- C ABI of the MI355X EntroPack library (libentropack.so).
 *
 * EntroPack (arXiv 2609.34185) stores a weight matrix W (R x C, C % 8 == 0)
 * as row-normalised E8 lattice points written as integer fields
 * (c, z1..z7, m) and coded with 32-state interleaved rANS in independently
 * decodable tiles (Sections 3.2-3.6, Appendix C.3).  This library provides
 *   - a CPU encoder (ep_encode_cpu) and the same encoder with its bulk passes
 *     on the GPU (ep_encode_gpu),
 *   - validation/inspection of an encoded blob on the host (ep_blob_info),
 *   - fused GPU decode on gfx950: rANS symbol decode with the coset-conditional
 *     tables, field inverse, row rescale and dtype snap, with no intermediate
 *     symbol tensor (ep_decode_tiles, ep_decode_layers; Section 3.7), for
 *     prepared layer stacks (ep_stack_prepare, ep_stack_decode) and for
 *     callers that cannot allocate (ep_decode_layers_noalloc),
 *   - an INT8 MFMA matrix product for decode-then-GEMM (ep_gemm_i8_nt),
 *   - decode fused with the matrix product, the decoded weights never written
 *     as a whole (ep_decode_matmul_i8 for a few int8 rows of X;
 *     ep_decode_gemm_i8 and ep_decode_gemm_bf16 on the matrix cores for any
 *     number of rows; App. D).
 *
 * Conventions shared by every entry point:
 *   - Return value: EP_OK (0) or a negative ep_status.  ep_last_error() gives a
 *     thread-local message for the last failing call on the calling thread.
 *     No C++ exception crosses this ABI.
 *   - "d_" pointers are device pointers (hipMalloc'd or equivalent) on the
 *     current HIP device; all other pointers are host pointers.
 *   - GPU calls are asynchronous on the given hipStream_t (passed as void*,
 *     NULL = default stream).  They allocate no device memory and never
 *     synchronise; the caller owns every buffer.  The exceptions are the GPU
 *     encoder (ep_encode_gpu), which allocates its work buffers and returns a
 *     finished host blob, and the preparation calls (ep_stack_prepare,
 *     ep_decode_gemm_i8_prepare, ep_decode_gemm_bf16_prepare), which return
 *     once their table build on the stream has completed.
 *   - Outputs must not alias the blob or each other.
 *
 * Stored representation (all little-endian; every section starts on a 4-byte
 * boundary; offsets in bytes from the start of the blob):
 *   header   48 B : u32 magic "EPK1", u32 version 1, u32 R, u32 C, u32 b,
 *                   u32 V (vectors per tile), u32 n_tiles, u32 container,
 *                   u32 table_bytes, u32 payload_words, u64 total_bytes
 *   tables        : u16 f0, u16 f1 (coset frequencies), then for coset
 *                   c = 0,1 and field i = 1..8 (z1..z7, m):
 *                   i32 min, u32 A, u16 f[A], padded to 4 B
 *   sigma         : f32[R]   row reconstruction scales (Section 3.5)
 *   delta         : f32[R]   container dequant scales (containers only)
 *   states        : u32[n_tiles][32] terminal rANS states (Appendix C.3)
 *   offsets       : u32[n_tiles + 1] payload offsets in 16-bit words
 *   payload       : u16[payload_words], padded to 4 B
 * Tile t holds vectors [tV, min((t+1)V, R*C/8)) (vector v = elements
 * 8v..8v+7 of the row-major matrix); tile-local vector i is coded by lane
 * i mod 32; each lane codes its vectors in order as [c, z1..z7, m]; the
 * decoder consumes words in (step ascending, lane ascending) order.
 */
#ifndef ENTROPACK_H
#define ENTROPACK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status, dtypes, containers ----------------------------------------- */
enum ep_status {
  EP_OK = 0,
  EP_ERR_ARG = -1,         /* invalid argument (shape, pointer, range, dtype) */
  EP_ERR_FORMAT = -2,      /* blob fails validation */
  EP_ERR_UNSUPPORTED = -3, /* valid request the library does not handle */
  EP_ERR_NOMEM = -4,       /* host allocation failed (encoder only) */
  EP_ERR_HIP = -5,         /* a HIP runtime call failed (launch error) */
  EP_ERR_CORRUPT = -6      /* decoded stream inconsistent (terminal state/offset) */
};

enum ep_dtype {
  EP_BF16 = 1,             /* round to nearest even, saturating at +-max finite */
  EP_FP16 = 2,             /* round to nearest even incl. subnormals, saturating at +-65504 */
  EP_FP32 = 3,             /* the FP32 product itself */
  EP_FP8_E4M3 = 4,         /* OCP e4m3fn, nearest even incl. subnormals, saturating at +-448 */
  EP_INT8 = 5,             /* clamp(round-half-even(y), -128, 127) */
  EP_FP8_E5M2 = 6,         /* OCP e5m2, nearest even incl. subnormals, saturating at +-57344 */
  EP_UINT8 = 7,            /* clamp(round-half-even(y), 0, 255) */
  EP_COORD2_I32 = 100      /* debug: the doubled lattice coordinates 2p as int32 */
};

enum ep_container {
  EP_CONT_DIRECT = 0,      /* the input values are coded directly */
  EP_CONT_FP8_ROW = 1,     /* row-scaled FP8 e4m3fn container (Appendix A.6, B.1) */
  EP_CONT_INT8_ROW = 2,    /* row-scaled symmetric INT8 container (Appendix B.1) */
  EP_CONT_FP8E5M2_ROW = 3, /* row-scaled FP8 e5m2 container (the dtype table of App. A.6) */
  EP_CONT_UINT8_TENSOR = 4 /* UINT8 with one scale per tensor and offset 128 (same table):
                              codes clamp(RNE(W/delta), -127, 127) + 128, delta = amax/127,
                              stored for every row; weights are delta * (value - 128) */
};

/* Bits of *d_status set by the decode kernels (OR-ed; the caller zeroes it). */
enum ep_status_bits {
  EP_STATUS_PAYLOAD_OVERRUN = 1,  /* a tile tried to read past its payload window */
  EP_STATUS_BAD_FINAL_STATE = 2,  /* a terminal state was not 2^15 after decoding */
  EP_STATUS_BAD_END_OFFSET = 4    /* a tile ended before its successor's offset */
};

/* ---- encoder ------------------------------------------------------------- */
typedef struct {
  double target_bpp;        /* requested stored rate R_tgt in bits per weight (> 0) */
  int32_t tile_vectors;     /* V: vectors per tile (>= 1); 512 = 4096 weights */
  int32_t prob_bits;        /* b0: 0 = 11 if target <= 7 else 12 (App. C.1); else 9..15 */
  int32_t search_steps;     /* geometric bisection steps I_s (App. C.1: 12) */
  int32_t container;        /* ep_container */
  double scale_lo, scale_hi;/* initial bracket of s (App. C.1: 1e-3, 8) */
  int64_t sample_vectors;   /* nominal sample size in 8-vectors (App. C.1: 2^18) */
  double state_credit_bits; /* bits credited per terminal state in eq. estimate (8) */
  int32_t nthreads;         /* worker threads, 0 = hardware concurrency */
  int32_t rdo_candidates;   /* K of the per-row rate-distortion refinement (Section 3.5,
                               App. C.2); <= 1 = off (default); at most 64 */
  int32_t rdo_sweeps;       /* T allocation sweeps of that refinement; 0 = off (default) */
  int32_t reserved;
} ep_encode_params;

typedef struct {
  uint8_t* data;            /* malloc'd by ep_encode_cpu; release with ep_blob_free */
  uint64_t size;
} ep_blob;

typedef struct {
  double scale;             /* selected quantisation scale s */
  double rate_estimate_sample; /* R_hat_sub at the last search step */
  double rate_stored;       /* R_stored = 8 B_stored / N (eq. objective) */
  double code_length_bits;  /* C_CE of the final tables on the full tensor */
  double erel_coded;        /* E_rel vs the coded values (container units for containers) */
  double erel_original;     /* E_rel vs the original input */
  double mean_state_bits;   /* mean log2(x_T / 2^15) over terminal states */
  uint64_t bytes;           /* blob size */
  uint64_t payload_bits;
  uint32_t prob_bits;       /* final b */
  uint32_t n_tiles;
  uint32_t max_alphabet;    /* largest field-table index range */
  uint32_t sample_rows;
  uint32_t escalations;     /* precision increases */
  uint32_t coarsenings;     /* coarsening steps after b = 15 */
  uint32_t rdo_rows_moved;  /* rows the refinement moved off the baseline scale */
  uint32_t reserved;
} ep_encode_stats;

/* Default parameters of the paper (App. C.1) with V = 512 and 8 credited bits. */
void ep_encode_params_default(ep_encode_params* p);

/* Encode W (R x C row-major; w_dtype EP_BF16 / EP_FP16 bit patterns or EP_FP32)
 * at p->target_bpp (Section 3.1 objective; Alg. rate selection in 3.4; refit
 * 3.5; optional per-row refinement, Section 3.5 and App. C.2, when
 * rdo_candidates > 1 and rdo_sweeps > 0; rANS 3.6).  On success out->data holds the blob (caller frees with
 * ep_blob_free) and *stats (nullable) is filled.  The output is independent of
 * nthreads.  Errors: EP_ERR_ARG (C % 8 != 0, R or C <= 0, non-finite input,
 * target <= 0, bad parameters), EP_ERR_NOMEM. */
int ep_encode_cpu(const void* w, int w_dtype, int64_t rows, int64_t cols,
                  const ep_encode_params* params, ep_blob* out, ep_encode_stats* stats);

/* The same encoder with its bulk passes on the GPU (quantisation, counts,
 * refit sums, rANS, statistics; the scale search and table normalisation run
 * on the host between passes).  d_w is a device array (R x C, same dtypes);
 * the result is a host blob byte-identical to ep_encode_cpu's for the same
 * inputs and parameters (nthreads is ignored), and *stats (nullable) equal to
 * its statistics (erel_coded and erel_original to rounding: their row sums
 * are taken in a different order).  Unlike the decode entry points it allocates device scratch
 * (about 10 bytes per weight for the values, fields and rANS words) and frees
 * it before returning, and it synchronises hip_stream: on return the blob is
 * complete.  Errors: as ep_encode_cpu, plus EP_ERR_HIP (device allocation or
 * launch failure) and EP_ERR_UNSUPPORTED (R >= 2^31).  The per-row refinement
 * holds rdo_candidates field sets on the device (4.5 bytes per weight each). */
int ep_encode_gpu(const void* d_w, int w_dtype, int64_t rows, int64_t cols,
                  const ep_encode_params* params, ep_blob* out, ep_encode_stats* stats,
                  void* hip_stream);
void ep_blob_free(ep_blob* blob);

/* ---- inspection ---------------------------------------------------------- */
typedef struct {
  uint32_t rows, cols, prob_bits, tile_vectors, n_tiles, container;
  uint32_t table_bytes, payload_words;
  uint64_t total_bytes;
  uint64_t off_tables, off_sigma, off_delta, off_states, off_offsets, off_payload;
  /* derived by ep_blob_info for kernel selection */
  uint32_t max_alphabet;     /* largest field-table index range A */
  int32_t coord2_min;        /* smallest doubled coordinate value any table can produce */
  int32_t coord2_max;        /* largest one */
  float max_abs_weight;      /* upper bound of |fp32(sigma_r * p)| over the tensor */
  uint32_t path;             /* decode kernel family chosen for this tensor: 1 narrow slot
                                table, 3 wide slot table, 2 bucketed search (all in LDS), 4
                                global tables (frequencies read from the blob in global
                                memory, App. C.3), the first that holds the tables; every
                                valid blob has one.  A caller may name another path that
                                holds the tables (any such path decodes the same bits). */
  uint32_t sum_alphabet;     /* sum of the field tables' index ranges */
  uint32_t table_off[16];    /* byte offset of field table 1 + 8c + (i-1) in the blob */
  int32_t table_min[16];     /* its min value */
  uint32_t table_A[16];      /* its index range */
  uint32_t coset_f0, coset_f1;
} ep_tensor_info;

/* Validate a host copy of a blob (n bytes) and fill *info: magic/version,
 * section bounds against n, n_tiles = ceil(R*C/8 / V), monotone offsets
 * ending at payload_words, every field table's frequencies summing to 2^b
 * with A <= 2^b, coset frequencies summing to 2^b, 9 <= b <= 15, finite
 * scales.  The device copy of the blob must be byte-identical.
 * Errors: EP_ERR_ARG (NULL), EP_ERR_FORMAT. */
int ep_blob_info(const void* host_blob, uint64_t n, ep_tensor_info* info);

/* ---- GPU decode ---------------------------------------------------------- */
/* Work mapping (every decode entry point): a wave decodes four tiles at a time
 * (two interleaved rANS chains, each over two tiles).  A launch with fewer than
 * 2048 such tasks whose layers all take the same slot-table path at b = 11 runs
 * two-tile tasks instead (one chain per wave): small layers then spread over
 * twice as many waves.  The environment variable EP_SMALL_TASK_LIMIT, read at
 * each call, replaces the 2048 (0: always four-tile tasks).  The outputs do
 * not depend on the choice. */
/* Decode tiles [tile_begin, tile_end) of one tensor (Section 3.7: eq.
 * rans_decode, eq. point_inverse, eq. recon).  d_out receives R x C
 * elements of out_dtype (row-major); only the elements of the given tiles are
 * written.  For containers, d_dequant (R floats, required; ignored for other
 * tensors) receives delta_r for each row whose first vector lies in a decoded
 * tile.  d_status (nullable, device
 * int32, zeroed by the caller) receives ep_status_bits for corrupt streams;
 * the kernels never read or write outside the blob's tile windows and the
 * output.  Errors (host side, before launch): EP_ERR_ARG (also for an info whose
 * path cannot hold the tensor's tables), EP_ERR_UNSUPPORTED, EP_ERR_HIP. */
int ep_decode_tiles(const ep_tensor_info* info, const void* d_blob, int out_dtype, void* d_out,
                    float* d_dequant, uint32_t tile_begin, uint32_t tile_end, int32_t* d_status,
                    void* hip_stream);

/* Fused decode and small-batch product (the decode of Section 3.7 feeding an
 * INT8 matrix product directly, the fusion the paper's conclusion leaves to
 * future work, on the INT8 route of Appendix B.1):
 *   Y[t][r] = sum_j X[t][j] * W'[r][j]   for t < m, r < R,
 * where W' is the tensor's INT8 container matrix exactly as ep_decode_tiles
 * writes it with EP_INT8 (the weights are delta_r * W'), X is m x C int8
 * row-major and Y m x R int32 row-major, exact (no rounding, no overflow:
 * C <= 131071).  W' is never written to memory: every decoded vector goes
 * straight into dot products with the m rows of X.  Y is overwritten (cleared
 * on hip_stream first by a small fill kernel, not a memset node, so the call
 * can be captured in a graph); d_dequant (R floats, required) receives delta_r
 * for every row.
 * All pointers are device memory owned by the caller; X 8-byte aligned.
 * Asynchronous on hip_stream, no allocation, one clear and one kernel launch.
 * d_status as for ep_decode_tiles.  Meant for few rows of X (decode-time
 * serving; it beats decode-then-GEMM up to about 4 rows); for more rows
 * decode once and call ep_gemm_i8_nt.
 * Errors: EP_ERR_ARG (null pointers, m outside 1..8), EP_ERR_UNSUPPORTED (not
 * the INT8 row container, C > 131071), EP_ERR_HIP. */
int ep_decode_matmul_i8(const ep_tensor_info* info, const void* d_blob, const int8_t* d_x, int m,
                        int32_t* d_y, float* d_dequant, int32_t* d_status, void* hip_stream);

/* Fused decode and MFMA product for any number of rows of X (the fusion of
 * Section 3.7's decode with the matrix product that the paper leaves to future
 * work, App. D; the decode-time cost it measures against the product's size in
 * App. A.5, Fig. cost; the INT8 route of App. B.1):
 *   Y[t][r] = sum_j X[t][j] * W'[r][j]   for t < m, r < R,
 * with W' the tensor's INT8 container matrix exactly as ep_decode_tiles writes it
 * with EP_INT8, X m x C int8 row-major, Y m x R int32 row-major, exact (C <=
 * 131071).  W' is never written as a whole: each workgroup decodes the tiles
 * touching a block of ceil(R / CUs) rows into its slab of d_workspace (the
 * block's rows plus a tile's reach on either side, so it stays in L2 and the
 * last-level cache) and multiplies X by those rows on the matrix cores
 * (v_mfma_i32_16x16x64_i8).  d_workspace: >= ep_decode_gemm_i8_workspace(info)
 * bytes of device memory owned by the caller, untouched until the launch
 * completes.  Y is overwritten (cleared first on hip_stream by a small fill
 * kernel whenever partial sums over K are added with atomics: at fewer rows of
 * X than 16 work items need, 256 to 976 rows by the block's height).
 * d_dequant (R floats, required) receives delta_r for every row; d_status as
 * for ep_decode_tiles.  Asynchronous, no allocation, at most one clear and one launch.
 * Errors: EP_ERR_ARG (null pointers, m outside 1..65536, X above 2^31 bytes, short
 * workspace), EP_ERR_UNSUPPORTED (not the INT8 row container, C > 131071),
 * EP_ERR_HIP. */
int ep_decode_gemm_i8(const ep_tensor_info* info, const void* d_blob, const int8_t* d_x, int64_t m,
                      int32_t* d_y, float* d_dequant, void* d_workspace, uint64_t ws_bytes,
                      int32_t* d_status, void* hip_stream);

/* Workspace bytes ep_decode_gemm_i8 and ep_decode_gemm_i8_prepared need for a
 * tensor on the current device: a 128 KiB area for the prepared decode tables, a
 * layer descriptor, then one slab per workgroup (0 if info is null or no device
 * is present). */
uint64_t ep_decode_gemm_i8_workspace(const ep_tensor_info* info);

/* Build the tensor's decode tables (the stage model of Section 3.7, the same
 * tables every workgroup of ep_decode_gemm_i8 builds in LDS) once, into the
 * table area of d_workspace, for later ep_decode_gemm_i8_prepared calls: the
 * serving case, where one weight is multiplied by new rows of X at every step.
 * d_workspace: >= ep_decode_gemm_i8_workspace(info) bytes of device memory
 * owned by the caller.  Synchronous: returns after the descriptor copy and the
 * table-building launch on hip_stream have completed.
 * Errors: as ep_decode_gemm_i8 (EP_ERR_ARG for a short workspace). */
int ep_decode_gemm_i8_prepare(const ep_tensor_info* info, const void* d_blob, void* d_workspace,
                              uint64_t ws_bytes, void* hip_stream);

/* ep_decode_gemm_i8 on a workspace that ep_decode_gemm_i8_prepare filled for this
 * same blob (d_blob unchanged since, workspace not used for another tensor in
 * between): every workgroup copies the prepared tables into LDS instead of
 * building them.  Same arguments, results and errors as ep_decode_gemm_i8; a
 * workspace prepared for another blob gives undefined values in Y (reads and
 * writes stay within the blob, X, Y, d_dequant and the workspace). */
int ep_decode_gemm_i8_prepared(const ep_tensor_info* info, const void* d_blob, const int8_t* d_x,
                               int64_t m, int32_t* d_y, float* d_dequant, void* d_workspace,
                               uint64_t ws_bytes, int32_t* d_status, void* hip_stream);

/* The same fused decode and MFMA product with BF16 operands, for any blob:
 *   Y[t][r] = sum_j X[t][j] * W'[r][j]   for t < m, r < R,
 * with W' the tensor exactly as ep_decode_tiles writes it with EP_BF16 (for
 * containers: the container values, the weights being delta_r * W'), X m x C
 * bf16 row-major (d_x), Y m x R fp32 row-major (d_y).  Each workgroup decodes
 * its block's tiles to bf16 in its slab and multiplies on the matrix cores
 * (v_mfma_f32_16x16x32_bf16); every product of two bf16 values is exact in
 * fp32 and the sums are fp32, so |Y - X W'^T| <= (C + s + 2) 2^-24 sum_j
 * |X[t][j] W'[r][j]| with s <= 16 partial sums per element (K is split over
 * waves at small m, as for the INT8 product, and those partial sums are added
 * with float atomics, so the last bits of Y may differ from call to call).
 * d_workspace: >= ep_decode_gemm_bf16_workspace(info) bytes.  Y is
 * overwritten (cleared first when K is split).  d_status as for
 * ep_decode_gemm_i8; d_dequant (R floats) receives delta_r for container
 * tensors (required for them, ignored otherwise).  Asynchronous,
 * no allocation, at most one clear and one launch.
 * Errors: EP_ERR_ARG (null pointers, m outside 1..65536, X above 2^31 bytes,
 * short workspace), EP_ERR_UNSUPPORTED, EP_ERR_HIP. */
int ep_decode_gemm_bf16(const ep_tensor_info* info, const void* d_blob, const void* d_x, int64_t m,
                        float* d_y, float* d_dequant, void* d_workspace, uint64_t ws_bytes,
                        int32_t* d_status, void* hip_stream);

/* Workspace bytes of ep_decode_gemm_bf16 (slabs hold bf16 rows; 0 if info is
 * null or no device is present). */
uint64_t ep_decode_gemm_bf16_workspace(const ep_tensor_info* info);

/* ep_decode_gemm_i8_prepare and ep_decode_gemm_i8_prepared for the BF16
 * product: the tables are built once into the workspace's table area, then
 * every ep_decode_gemm_bf16_prepared call copies them (same contract). */
int ep_decode_gemm_bf16_prepare(const ep_tensor_info* info, const void* d_blob, void* d_workspace,
                                uint64_t ws_bytes, void* hip_stream);
int ep_decode_gemm_bf16_prepared(const ep_tensor_info* info, const void* d_blob, const void* d_x,
                                 int64_t m, float* d_y, float* d_dequant, void* d_workspace,
                                 uint64_t ws_bytes, int32_t* d_status, void* hip_stream);

/* One layer of a stack decode. */
typedef struct {
  ep_tensor_info info;       /* from ep_blob_info on the host copy */
  const void* d_blob;
  void* d_out;
  float* d_dequant;          /* R floats, required for container tensors, else ignored */
  int32_t out_dtype;
  int32_t reserved;
} ep_layer;

/* Workspace bytes ep_decode_layers needs for n layers (device memory): 0 for
 * n <= 8 (the descriptors travel as kernel arguments), else n descriptors. */
uint64_t ep_decode_layers_workspace(int n);

/* Decode every tile of n layers with a single kernel launch.  Up to 8 layer descriptors are passed as kernel
 * arguments; longer lists are copied into d_workspace (>=
 * ep_decode_layers_workspace(n) bytes, device memory owned by the caller) by
 * one hipMemcpyAsync on the same stream, which has read the host list by the
 * time it returns; d_workspace must stay untouched until the launch completes.
 * Layers may take different decode paths (ep_tensor_info.path): each
 * workgroup builds the tables of the layer it works on in that layer's form.
 * The layers array is host memory and is not retained.  Errors: as
 * ep_decode_tiles, and EP_ERR_ARG for a missing or short workspace. */
int ep_decode_layers(const ep_layer* layers, int n, void* d_workspace, uint64_t ws_bytes,
                     int32_t* d_status, void* hip_stream);

/* The same decode as ep_decode_layers for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): no workspace argument and no allocation of any kind.  The layer
 * descriptors are copied (one hipMemcpyAsync on hip_stream, which has read the host
 * list when it returns) into a static device array of the library, 512 descriptors
 * in size, that each device keeps until the process ends; n above 512 is refused
 * with EP_ERR_ARG.  Every call on a device shares that array: calls that overlap on
 * one device (several streams, several host threads) race and must be serialised by
 * the caller; consecutive calls on one stream are ordered.  Errors: as
 * ep_decode_layers, and EP_ERR_HIP when the array's address cannot be found. */
int ep_decode_layers_noalloc(const ep_layer* layers, int n, int32_t* d_status, void* hip_stream);

/* ---- prepared stacks ------------------------------------------------------ */
/* A layer list whose device descriptors and decode tables were written once by
 * ep_stack_prepare, so that every later decode of the same blobs into the same
 * outputs (one per forward pass of a compressed model) is a single kernel launch
 * with no copy: its workgroups load each layer's prepared tables instead of
 * rebuilding them from the blob. */
typedef struct {
  void* d_workspace;         /* device descriptor list (caller-owned memory) */
  int32_t n_layers;
  uint32_t path;             /* decode path shared by all layers, or 15 for a list of several */
  uint32_t total_tasks;      /* 4-tile tasks over all layers */
  uint32_t lds_bytes;        /* LDS of the launch */
  uint32_t reserved[4];
} ep_stack;

/* Device bytes ep_stack_prepare needs for n layers: the descriptors and one
 * 128 KiB decode-table image per layer. */
uint64_t ep_stack_workspace(int n);

/* Validate n layers (as for ep_decode_layers), write their descriptors and build
 * their decode tables into d_workspace (>= ep_stack_workspace(n) bytes, device
 * memory owned by the caller, which must outlive every ep_stack_decode of this
 * stack; the blobs must stay unchanged too) and fill *stack.  Synchronous:
 * returns after the copy and the table-building launch on hip_stream have
 * completed.
 * Errors: as ep_decode_layers, EP_ERR_ARG for a null stack or short workspace. */
int ep_stack_prepare(const ep_layer* layers, int n, void* d_workspace, uint64_t ws_bytes,
                     ep_stack* stack, void* hip_stream);

/* Decode every tile of a prepared stack: one kernel launch on hip_stream, no
 * host-to-device copy, no allocation.  d_status as for ep_decode_tiles.
 * Errors: EP_ERR_ARG for an unprepared stack, EP_ERR_UNSUPPORTED, EP_ERR_HIP. */
int ep_stack_decode(const ep_stack* stack, int32_t* d_status, void* hip_stream);

/* ---- decode-then-GEMM ---------------------------------------------------- */
/* Y[M x N] (int32, row-major) = A[M x K] (int8, row-major) * B[N x K]^T
 * (int8, row-major: both operands K-contiguous) on MFMA, exact int32
 * accumulation: the product of decoded INT8 weights (B) with INT8
 * activations, as in the compressed-storage INT8 route of the paper's
 * Appendix B.1.  All pointers are device memory owned by the caller; A and B
 * 16-byte aligned.  Requires M, N > 0, K > 0, K % 16 == 0 and K <= 131071 (each
 * product is at most 2^14 in magnitude, so every int32 sum is exact).
 * Y is overwritten whatever it held.  A launch of few 256 x 256 tiles (at
 * most half as many as CUs, e.g. few rows of A) splits K over several
 * workgroups per tile: a small fill kernel clears Y first and the partial
 * sums are added with atomics (exact, order-independent); calls that overlap
 * on the same Y then race.  Asynchronous on hip_stream, no allocation, no
 * memset node (graph capture is safe).  Errors: EP_ERR_ARG, EP_ERR_HIP. */
int ep_gemm_i8_nt(const int8_t* d_a, const int8_t* d_b, int32_t* d_y, int64_t m, int64_t n,
                  int64_t k, void* hip_stream);

/* ---- errors -------------------------------------------------------------- */
const char* ep_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
