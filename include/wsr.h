/*
 * wsr.h - weight-streaming read kernels for AMD Instinct MI355X (gfx950): the C ABI.
 *
 * The operations are the ones "The Ingestion Tax: Adopting File-Backed Weights in Tensor
 * Frameworks" measures: a batch-1 decode step rereads every weight byte once per token (Sec. 1,
 * Sec. 6.2), the single-token GEMV of the matched protocol (Sec. 3.1), the pure-read reference that
 * sets its ceiling (Sec. 3.1, Sec. 3.3), and the same kernels over host pages mapped into the GPU's
 * address space (Sec. 5.1, Alg. 1; Sec. 7.3 for a discrete GPU on PCIe).
 *
 * Conventions shared by every entry point:
 *  - Each call returns a wsr_status.  Arguments are checked before anything is enqueued: on any
 *    status other than WSR_OK nothing was enqueued, except WSR_E_HIP from a failed kernel launch,
 *    which may follow launches the same call already made.  A message for the calling thread is
 *    available from wsr_last_error().  No call aborts or exits.
 *  - Compute calls only enqueue work on the caller's HIP stream (`stream` is a hipStream_t; NULL
 *    means the null stream of the current device) and return without waiting for the device: the
 *    execution contract's C3, ordering on the GPU with no host drain (Sec. 2.2, Table 1).  Results
 *    stay in device-visible memory (C2).  Kernels run on the current HIP device, which must be the
 *    stream's device.
 *  - The library never allocates, frees or retains caller memory.  Every pointer is caller-owned and
 *    must stay valid until the stream has passed the enqueued work.  Weights and inputs are only
 *    read (`const`); the library writes only the outputs (y, *sum_dev) and the workspace (ws).
 *  - Device pointers may point to HBM or to host memory made device-visible (see
 *    wsr_register_host); the kernels are the same either way.
 *  - Sizes are element counts unless a name ends in `_bytes`.  Matrices are row-major (M, K) with
 *    strides (K, 1), as in Alg. 1.
 *  - Results are deterministic: a given input and shape always gives bitwise-identical output,
 *    whatever memory the operands live in.
 *  - Not thread-safe per workspace: concurrent calls must use distinct workspaces.
 */
#ifndef WSR_H
#define WSR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WSR_ABI_VERSION 3

typedef enum {
    WSR_OK = 0,
    WSR_E_ARG = 1,          /* null pointer, negative size, unknown format or flag, n_tokens < 1  */
    WSR_E_ALIGN = 2,        /* host range base or length not a page multiple (Alg. 1's reject
                               rule); device operand misaligned; K % 8 != 0 (16-bit) or
                               K % 32 != 0 (q4) or K % 16 != 0 (int8)                            */
    WSR_E_SIZE = 3,         /* workspace too small, or a size whose byte count overflows        */
    WSR_E_UNSUPPORTED = 4,  /* the runtime refused a request, e.g. pinning an existing host range
                               (distinct from a failed HIP call, Sec. 7.3)                      */
    WSR_E_STATE = 5,        /* range already registered, or unregister of an unknown range      */
    WSR_E_HIP = 6           /* a HIP runtime call or kernel launch failed                       */
} wsr_status;

typedef enum {
    WSR_F16 = 1,    /* IEEE binary16                                                          */
    WSR_BF16 = 2,   /* bfloat16                                                               */
    WSR_Q4 = 3,     /* blocks of 32 signed int4 weights sharing one fp16 scale (see gemv_q4)   */
    WSR_I8 = 4      /* signed int8 weights with one fp16 scale per row (see gemv_i8)           */
} wsr_fmt;

/* Message describing the last failed call on this thread ("" if none). */
const char* wsr_last_error(void);

/* WSR_ABI_VERSION of the library actually loaded. */
int wsr_abi_version(void);

/* ---- host memory read in place -------------------------------------------------------------

   wsr_register_host: make host range [host, host + bytes) readable by the kernels and return its
   device address.  Follows the producer of Alg. 1 (Sec. 5.1): the range must start on a page
   boundary and its length must be a whole number of pages (else WSR_E_ALIGN: a partial page would
   alias a neighbouring tensor); one call yields one registration and nothing is cached by address
   (WSR_E_STATE if [host] is already registered).
   - A range already device-visible (pinned host memory from hipHostMalloc, e.g. a PyTorch pinned
     tensor) is adopted in place: no copy and no new pin; *granted_out gets WSR_REG_PREPINNED.  The
     whole range must lie inside that one pinned allocation (WSR_E_SIZE if it runs past its end;
     WSR_E_UNSUPPORTED if the runtime does not report the allocation's extent).
   - Any other range is pinned with hipHostRegister only if `flags` has WSR_REG_PIN; with
     WSR_REG_READONLY as well, a read-only pin is requested first (Sec. 5.1, read-only intent) and
     *granted_out reports WSR_REG_READONLY if it was granted.  A refused pin returns
     WSR_E_UNSUPPORTED: registration and direct read are separate capabilities (Sec. 7.3).  Without
     WSR_REG_PIN such a range returns WSR_E_UNSUPPORTED.  Map file pages MAP_SHARED: pinning a
     private mapping for write would turn file pages into anonymous copies (Sec. 5.3).
   - Synchronous; callable from any thread.  dev_out receives the device address; granted_out may
     be NULL. */
#define WSR_REG_READONLY 1u     /* request: read-only mapping       | granted: read-only       */
#define WSR_REG_PIN 2u          /* request: pin a range not yet device-visible                 */
#define WSR_REG_PREPINNED 4u    /* granted: range was already device-visible, adopted in place  */
wsr_status wsr_register_host(const void* host, size_t bytes, unsigned flags, const void** dev_out,
                             unsigned* granted_out);

/* Release the registration made for `host` (unpins only what wsr_register_host pinned).  Call it
   after the last kernel reading the range has completed and before unmapping the range (Alg. 1's
   deleter order: release the GPU view, then unmap).  WSR_E_STATE if `host` is not registered. */
wsr_status wsr_unregister_host(const void* host);

/* ---- streaming-read probe --------------------------------------------------------------------

   *sum_dev = sum over i < n of buf[i], accumulated in fp64: the pure-read reference that streams
   every byte once with no other arithmetic (Sec. 3.1, Sec. 3.3).  Each block sums a contiguous
   part of the buffer into an fp64 partial in the workspace; a second launch adds the partials in
   index order.  The result stays in device memory.
   buf: fp32, 16-byte aligned, device-visible; n >= 0 (n = 0 gives 0).  sum_dev: one fp64,
   device memory.  ws: at least wsr_probe_workspace_bytes(n) bytes of device memory, 16-byte
   aligned (its contents need no initialisation). */
size_t wsr_probe_workspace_bytes(size_t n);
wsr_status wsr_probe_read(const float* buf, size_t n, double* sum_dev, void* ws, size_t ws_bytes,
                          void* stream);

/* ---- single-token GEMVs (Sec. 3.1: one token, one weight read per byte) ------------------------

   wsr_gemv_f16: y[i] = sum_k W[i*K + k] * x[k] for i < M, with W and x both fp16 (fmt WSR_F16) or
   both bf16 (WSR_BF16), products and sums in fp32, y fp32.
   W: (M, K) row-major, 16-byte aligned; x: K elements, 16-byte aligned; y: M floats, 4-byte
   aligned.  M >= 0, K >= 0, K % 8 == 0 (K = 0 gives y = 0). */
wsr_status wsr_gemv_f16(const void* W, const void* x, float* y, int64_t M, int64_t K, int fmt,
                        void* stream);

/* wsr_gemv_q4: y[i] = sum_k w[i,k] * x[k] with w[i,k] = q[i,k] * s[i, k/32].
   Wq: uint8 (M, K/2), byte j of row i holds q[i,2j] in its low nibble and q[i,2j+1] in its high
   nibble, two's-complement int4 in -8..7; 16-byte aligned.  scales: fp16 bits (M, K/32), 2-byte
   aligned.  x: fp16[K], 16-byte aligned.  y: fp32[M].  K % 32 == 0.  Dequantised weights are
   exact (q * s needs 15 significant bits) and every product and sum is fp32. */
wsr_status wsr_gemv_q4(const uint8_t* Wq, const uint16_t* scales, const uint16_t* x, float* y,
                       int64_t M, int64_t K, void* stream);

/* wsr_gemv_i8: y[i] = s[i] * sum_k q[i,k] * x[k], the matched protocol's weight format (Sec. 3.1:
   int8 codes with fp16 row scales).  Wq: int8 (M, K) row-major, 16-byte aligned.  scales: fp16
   bits [M], 2-byte aligned.  x: fp16[K], 16-byte aligned.  y: fp32[M].  K % 16 == 0.  Every
   product q * x is exact in fp32 and sums are fp32; the row scale multiplies the finished sum. */
wsr_status wsr_gemv_i8(const int8_t* Wq, const uint16_t* scales, const uint16_t* x, float* y,
                       int64_t M, int64_t K, void* stream);

/* ---- multi-column GEMV (Sec. 3.4 and 5.2: T activation columns share each weight read) ---------

   wsr_gemv_f16_cols: for t < T and i < M, y_t[i] = sum_k W[i*K + k] * x_t[k], where
   x_t = x + t * x_col_stride bytes and y_t = y + t * y_col_stride bytes.  W, x_t and y_t follow
   wsr_gemv_f16's layout, formats and alignment; T is 1, 2, 4, 8 or 16; x_col_stride >= 0 and a
   multiple of 16 (0: every column reads the same x); y_col_stride a multiple of 4 and, for T > 1,
   at least 4 M so that the output columns do not overlap (else WSR_E_ARG).  Every y_t is
   bitwise equal to wsr_gemv_f16(W, x_t, y_t, M, K, fmt). */
wsr_status wsr_gemv_f16_cols(const void* W, const void* x, int64_t x_col_stride, float* y,
                             int64_t y_col_stride, int64_t M, int64_t K, int32_t T, int fmt,
                             void* stream);

/* wsr_gemv_q4_cols: the same for q4 weights (wsr_gemv_q4's layout), T = 1, 2, 4 or 8: each
   block is decoded once and used for every column.  Every y_t is bitwise equal to
   wsr_gemv_q4(Wq, scales, x_t, y_t, M, K). */
wsr_status wsr_gemv_q4_cols(const uint8_t* Wq, const uint16_t* scales, const uint16_t* x,
                            int64_t x_col_stride, float* y, int64_t y_col_stride, int64_t M, int64_t K,
                            int32_t T, void* stream);

/* wsr_gemv_i8_cols: the same for int8 weights (wsr_gemv_i8's layout), T = 1, 2, 4 or 8.  Every
   y_t is bitwise equal to wsr_gemv_i8(Wq, scales, x_t, y_t, M, K). */
wsr_status wsr_gemv_i8_cols(const int8_t* Wq, const uint16_t* scales, const uint16_t* x,
                            int64_t x_col_stride, float* y, int64_t y_col_stride, int64_t M, int64_t K,
                            int32_t T, void* stream);

/* ---- decode weight sweep ----------------------------------------------------------------------

   For t in [0, n_tokens), for m in [0, n) in order: y_m(t) = W_m . x_m(t), where
   x_m(t) = x + t * x_tok_stride bytes and y_m(t) = y + t * y_tok_stride bytes.  One batch-1 token
   reads every matrix once (Sec. 6.2) and a pass over all of them is ordered on the GPU with no
   host synchronisation (Sec. 3.1; C3 of Table 1).  Each matrix follows wsr_gemv_f16 (fmt WSR_F16
   or WSR_BF16), wsr_gemv_q4 (WSR_Q4) or wsr_gemv_i8 (WSR_I8), `scales` set for the last two, and
   their layout and alignment rules.
   Matrices of one token run in one persistent launch unless a matrix has WSR_MAT_AFTER_PREVIOUS,
   which starts a new launch so that it may read outputs of earlier matrices of the same token.
   ws: at least wsr_sweep_workspace_bytes(mats, n) bytes of device memory, 256-byte aligned; each
   call writes the launches' work counters, the matrix table and the matrices' stream offsets
   there (no initialisation needed). */
#define WSR_MAT_AFTER_PREVIOUS 1
typedef struct wsr_mat {
    int32_t fmt;            /* wsr_fmt                                                    */
    int32_t flags;          /* 0 or WSR_MAT_AFTER_PREVIOUS                                */
    int64_t M, K;
    const void* w;          /* weights (16-bit), packed int4 codes (q4) or int8 codes      */
    const void* scales;     /* q4 block scales or int8 row scales, NULL otherwise         */
    const void* x;          /* activation of token 0                                      */
    int64_t x_tok_stride;   /* bytes between tokens' activations (0: same x every token)  */
    float* y;               /* output of token 0                                          */
    int64_t y_tok_stride;   /* bytes between tokens' outputs                              */
} wsr_mat;

size_t wsr_sweep_workspace_bytes(const wsr_mat* mats, int32_t n);
wsr_status wsr_decode_sweep(const wsr_mat* mats, int32_t n, int32_t n_tokens, void* ws,
                            size_t ws_bytes, void* stream);

/* wsr_decode_sweep_batched: the same outputs as wsr_decode_sweep, bit for bit, with the tokens
   taken `batch` at a time (1, 2, 4, 8 or 16): one pass over the weights serves tokens
   t .. t + batch - 1, whose activations must all be ready when the call is made, as for a batch of
   independent sequences or the candidates of a speculative step (Sec. 3.4, 5.2).  The last
   n_tokens % batch tokens go in passes of the largest power of two that fits.  A table holding a
   q4 or int8 matrix is swept at most 8 tokens per pass (batch 16 acts as 8).  With batch > 1 every matrix
   must have y_tok_stride >= 4 M.  ws as for wsr_decode_sweep. */
wsr_status wsr_decode_sweep_batched(const wsr_mat* mats, int32_t n, int32_t n_tokens, int32_t batch,
                                    void* ws, size_t ws_bytes, void* stream);

/* ---- the decode sweep without a workspace ------------------------------------------------------

   wsr_decode_sweep_noalloc: for callers that cannot allocate device memory (code under HIP graph
   capture, tight serving loops, harnesses that forbid hipMalloc).  The outputs of
   wsr_decode_sweep(mats, n, n_tokens, ws, ws_bytes, stream), bit for bit (the same kernels), with
   the workspace taken from the library's own scratch: a device array of 512 KiB per GPU, which
   holds the table of up to about 5,000 matrices (wsr_sweep_workspace_bytes(mats, n) <= 524288,
   else WSR_E_SIZE; a 70B-shaped model has 561).  The call allocates and frees nothing.  The first
   call on a device looks up that device's scratch address (a HIP query, no allocation); the
   scratch stays with the device until the process ends.  Every call on one GPU shares that GPU's
   scratch, and each call rewrites it before use (table and counters; nothing carries over).
   Calls enqueued on one stream run one after another; calls whose work overlaps on one GPU (on
   different streams, or from several threads with no ordering between them) race on the scratch
   and must not be made. */
wsr_status wsr_decode_sweep_noalloc(const wsr_mat* mats, int32_t n, int32_t n_tokens, void* stream);

/* ---- batched decode on the matrix cores (Sec. 3.4, 5.2: several activation columns per weight read) -

   wsr_decode_sweep_mma: for t < n_tokens and every matrix m, y_m(t) = W_m . x_m(t) as in
   wsr_decode_sweep, with up to 16 tokens per pass over the weights and the products formed by the
   matrix cores (v_mfma_f32_16x16x32): each 16-row, 16-token tile accumulates slabs of 32 weights,
   used as stored for fp16 and bf16, decoded to exact fp16 integers for int8, and for q4 to the
   exact fp16 subnormals (q + 8) 2^-24 with the bias removed by one more matrix instruction per
   slab and the sums scaled back by 2^24.  Every product is exact and sums are fp32, but a slab's
   products are added in the matrix core's own order, so outputs agree with wsr_decode_sweep within
   rounding (not bit for bit: relative L2 within 1e-5 per matrix over 16 tokens on the tested
   models, up to about 1.2e-5 for single tokens of 14,336-long q4 rows); a unit activation vector
   still returns the dequantised weights exactly.  Tokens go in passes of 16, the
   last pass holding the rest.  A pass of a single token (n_tokens = 1, or a last pass of one) runs
   the vector-ALU loop of wsr_decode_sweep instead, whose outputs it then equals bit for bit: a
   matrix instruction would compute 16 token slots to use one.  Formats, layouts, flags and the workspace as for wsr_decode_sweep;
   with n_tokens > 1 every matrix must have y_tok_stride >= 4 M.  A row may hold at most 32 MiB of
   weights or codes and x_tok_stride may be at most 128 MiB (WSR_E_SIZE otherwise): the kernels
   address 64 rows and 16 tokens with 32-bit offsets. */
wsr_status wsr_decode_sweep_mma(const wsr_mat* mats, int32_t n, int32_t n_tokens, void* ws, size_t ws_bytes,
                                void* stream);

/* ---- ordering against a framework stream (execution contract C3, Table 1; Sec. 4.3) -----------

   wsr_decode_sweep_ordered: the outputs of wsr_decode_sweep, with the pass ordered after all work
   already enqueued on `framework_stream` and all later work on `framework_stream` ordered after the
   pass, by one of four mechanisms (Sec. 4.3 compares their cost under an in-flight workload):
     WSR_ORDER_STREAM      the pass is enqueued on framework_stream itself (own_stream unused);
     WSR_ORDER_EVENT       the pass runs on own_stream, which waits on the GPU for an event
                           recorded on framework_stream;
     WSR_ORDER_HOST_EVENT  as WSR_ORDER_EVENT, but the host waits for that event before it
                           enqueues the pass (the signal becomes host-visible; the call blocks);
     WSR_ORDER_DRAIN       the host drains the whole device (hipDeviceSynchronize) first.
   In the last three, framework_stream then waits on the GPU for an event recorded after the pass.
   Only WSR_ORDER_STREAM and WSR_ORDER_EVENT keep every dependency on the GPU.  Calls on one
   device are serialised while they enqueue (events shared per device). */
#define WSR_ORDER_STREAM 0
#define WSR_ORDER_EVENT 1
#define WSR_ORDER_HOST_EVENT 2
#define WSR_ORDER_DRAIN 3
wsr_status wsr_decode_sweep_ordered(const wsr_mat* mats, int32_t n, int32_t n_tokens, void* ws, size_t ws_bytes,
                                    void* framework_stream, void* own_stream, int32_t mode);

/* ---- per-use copy endpoint (Sec. 8.1; Table 2, pipelined double-buffered copy; Sec. 7.2,
   overlapped streaming) ---------------------------------------------------------------------

   wsr_sweep_staged: the outputs of wsr_decode_sweep for the single token `token`, bit for bit,
   with every matrix's weights (and scales) copied per use from wherever they live (pageable or
   pinned host memory, or device memory) into a device staging buffer instead of being read in
   place.  `stage` (device memory, 256-byte aligned) is split into two halves; each matrix goes in
   chunks of whole rows that fit a half (codes first, scales after them at a 256-byte boundary),
   alternating halves.  Copies run on `copy_stream` and GEMVs on `stream`: the copy of a chunk into
   a half waits for the GEMV that last read that half, and each GEMV waits for its chunk's copy,
   so the copy of chunk k + 1 overlaps the GEMV of chunk k.  The first copy waits for the work
   already enqueued on `stream`; on return, all work of the call is ordered before later work on
   `stream`.  Use distinct streams for overlap (the same stream also works, serially).  The source
   memory must stay valid and unchanged until the copies have run.  Pageable host sources go
   through two pinned host halves the library keeps per device (each the size of a stage half):
   host threads copy a chunk into one half while the previous chunk moves out of the other, so for
   such sources the call blocks until its last chunk is in a pinned half.  Chunks in pinned host
   pages (a bounce half, or a caller's matrix that lies wholly in one pinned allocation) with
   16-byte aligned ends are copied by a kernel of the library on copy_stream, which reads them
   across PCIe; other chunks by hipMemcpyAsync on copy_stream.  mats: as wsr_decode_sweep, except that w and scales may
   be host pointers; x and y device memory.  WSR_E_SIZE if half of stage_bytes, less 256, holds no
   row of some matrix.  Calls on one device are serialised while they enqueue (events shared per
   device). */
wsr_status wsr_sweep_staged(const wsr_mat* mats, int32_t n, int32_t token, void* stage, size_t stage_bytes,
                            void* stream, void* copy_stream);

/* ---- endpoint selection (Alg. 2, Sec. 8.1) -------------------------------------------------------

   wsr_host_resident_pages: how many of the pages spanning [host, host + bytes) are resident in
   memory (mincore), for Alg. 2's check that a prefaulted mapped set is resident and that it
   survives one pass of every arm (page-cache residency control, Table 5).  WSR_E_ARG if part of
   the range is not mapped. */
wsr_status wsr_host_resident_pages(const void* host, size_t bytes, size_t* resident_pages, size_t* total_pages);

/* wsr_select_endpoint: Alg. 2 over measured endpoint rates.  Path time is W / B per endpoint
   (Sec. 8.1).  In order: a mapped set that is not resident stops with WSR_EP_STORAGE_BOUND; the
   resident endpoint is dropped when resident_ok is 0 (its allocation failed, or the mapping was
   evicted after one pass of every arm); endpoints named in `excluded` (bit 1 << WSR_EP_x: import
   or capacity limits) or with rate <= 0 (not measured) are dropped; among the survivors the
   fastest wins, except that mapping wins whenever its time exceeds the fastest by at most
   theta (a fraction: 0.05 is the paper's 5 % band) of the fastest time.  *choice receives the
   endpoint (WSR_EP_NONE if none survives); times_ms, if not NULL, receives W / B in milliseconds
   for map, resident and copy (-1 where not measured). */
typedef enum {
    WSR_EP_NONE = 0,
    WSR_EP_MAP = 1,             /* read the file pages (host memory) in place                    */
    WSR_EP_RESIDENT = 2,        /* one copy into device memory, reused by every pass            */
    WSR_EP_COPY = 3,            /* per-use copy (wsr_sweep_staged)                               */
    WSR_EP_STORAGE_BOUND = 4    /* the mapped set is not resident: outside the studied regime   */
} wsr_endpoint;

typedef struct wsr_endpoint_probe {
    double w_bytes;             /* working set W (bytes)                                          */
    double rate[3];             /* B_map, B_resident, B_copy in bytes/s, measured with one kernel */
    int32_t mapped_resident;    /* every page of the mapped set resident after prefaulting        */
    int32_t resident_ok;        /* resident arm allocated and the mapping survived every arm     */
    uint32_t excluded;          /* endpoints dropped for import or capacity limits               */
    int32_t reserved;           /* 0                                                              */
} wsr_endpoint_probe;

wsr_status wsr_select_endpoint(const wsr_endpoint_probe* p, double theta, int32_t* choice, double* times_ms);

#ifdef __cplusplus
}
#endif
#endif /* WSR_H */
