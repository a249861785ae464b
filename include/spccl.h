/*
 * spccl.h -- C ABI of the MI355X (gfx950) Pici hot path of SpCCL
 * (arXiv 2607.04676): dense <-> Pici codec, elementwise reduction with
 * fill-in, gather-expand, and ring collectives over P virtual ranks held in
 * one GPU's memory.
 *
 * Conventions for every entry point:
 *  - Pointers are device pointers unless marked "host".  Messages and
 *    workspaces must be 16-byte aligned; dense arrays need only the alignment
 *    of their element type.  The caller owns every buffer; the library
 *    allocates and frees nothing.
 *  - `stream` is a hipStream_t handle (NULL = the default stream).  Calls are
 *    asynchronous on it, except spccl_read_header, spccl_read_status and the
 *    spccl_vr_* collectives, which synchronize it.
 *  - Errors found on the host (bad argument, capacity, size, dtype) are
 *    returned before anything is launched.  Data errors found on the device
 *    (a corrupt input message) set a sticky status word in the workspace `ws`
 *    (read it with spccl_read_status).  A message whose header fails its
 *    checks is not read and the call writes no output; a tile whose index
 *    entries disagree with its bit vector, or that sets a bit at a position
 *    >= n, is treated as empty.  After any
 *    device error, re-initialise the workspace before reusing it.
 *  - Element types: SPCCL_F32 (IEEE binary32) and SPCCL_BF16 (bfloat16),
 *    handled as raw bit patterns.  n < 2^32 per message (I is 32-bit).
 *  - An element is nonzero ("present") iff its bit pattern is not all zero,
 *    so -0.0 is kept and decompress(compress(x)) == x bit for bit.
 *  - NaN values are outside the contract of the reductions.
 */
#ifndef SPCCL_H
#define SPCCL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SPCCL_OK = 0,
    SPCCL_ERR_INVALID_ARG = 1,     /* null/unaligned pointer, bad enum, n % P != 0, ... */
    SPCCL_ERR_CAPACITY = 2,        /* an output buffer is smaller than required */
    SPCCL_ERR_UNSUPPORTED = 3,     /* dtype or size outside the supported range */
    SPCCL_ERR_CORRUPT_STREAM = 4,  /* a message failed its header / index checks */
    SPCCL_ERR_WORKSPACE = 5,       /* workspace too small or not initialised */
    SPCCL_ERR_HIP = 6,             /* a HIP runtime call or kernel launch failed */
    SPCCL_ERR_TIMEOUT = 7          /* a device-side wait exceeded its spin limit */
} spccl_status_t;

typedef enum { SPCCL_F32 = 0, SPCCL_BF16 = 1 } spccl_dtype_t;

/* Message formats (Sec. V-B: each message carries its format in its header).
 * COO is the flat variant of Sec. II-B that the paper runs beside Pici
 * (Sec. IV-D): one 32-bit index and one value per nonzero. */
typedef enum { SPCCL_FMT_DENSE = 0, SPCCL_FMT_PICI = 1, SPCCL_FMT_COO = 2 } spccl_format_t;

/* A reduce operand is either a raw dense array of n elements (ARRAY) or a
 * header-prefixed message (STREAM). */
typedef enum { SPCCL_ARRAY = 0, SPCCL_STREAM = 1 } spccl_kind_t;

typedef struct {
    int32_t kind;     /* spccl_kind_t */
    int32_t fmt;      /* spccl_format_t of a STREAM: for an input, the format the
                         caller expects (checked against the header on the device);
                         for an output, the format to produce.  Ignored for ARRAY. */
    void* ptr;        /* device pointer (16-byte aligned for a STREAM) */
    uint64_t bytes;   /* capacity of the buffer in bytes; a STREAM input must hold
                         at least the smallest valid message of its declared
                         format (DENSE: 48 + n * elem_size; PICI: off_A, the
                         header plus B and I; COO: the 48-byte header), else
                         SPCCL_ERR_CAPACITY */
} spccl_operand_t;

/* The 48-byte message header (Sec. V-B names its contents: format, size and
 * component offsets; the layout is this library's).  Little-endian.
 *   PICI:  B (u64[64*T]) at offset 48, I (u32[T+1]) at off_I = 48 + 512*T,
 *          zero pad to 16 bytes, A (nnz values) at off_A,
 *          total_bytes = off_A + nnz * elem_size.
 *   COO:   J (u32[nnz], the flat indices of the nonzeros, strictly
 *          increasing) at off_I = 48, zero pad to 16 bytes, V (nnz values in
 *          index order) at off_A = align16(48 + 4*nnz),
 *          total_bytes = off_A + nnz * elem_size.
 *   DENSE: the n values at off_A = 48; off_I = 0; nnz = UINT64_MAX
 *          ("not computed"); total_bytes = 48 + n * elem_size. */
typedef struct {
    uint32_t magic;        /* 0x49434950: the bytes "PICI" */
    uint16_t format;       /* spccl_format_t */
    uint16_t dtype;        /* spccl_dtype_t */
    uint64_t n;            /* elements represented */
    uint64_t nnz;          /* nonzeros (PICI) or UINT64_MAX (DENSE) */
    uint64_t off_I;
    uint64_t off_A;
    uint64_t total_bytes;  /* bytes of the whole message, header included */
} spccl_header_t;

#define SPCCL_MAGIC 0x49434950u
#define SPCCL_HEADER_BYTES 48u
#define SPCCL_NNZ_UNKNOWN UINT64_MAX

/* ---- sizes --------------------------------------------------------------- */

/* T = ceil(n / 4096): the 64x64 virtual tiles covering n elements (Sec. III-B). */
uint64_t spccl_num_tiles(uint64_t n);

/* Exact byte size of a Pici message with nnz nonzeros: the paper's component
 * sizes (B 512*T, I 4*(T+1), A nnz*s; Sec. III-B) plus header and pad. */
uint64_t spccl_pici_bytes(uint64_t n, int32_t dtype, uint64_t nnz);

/* Worst-case message size for n elements (every element present).  Every
 * message output must have at least this capacity, because the size is only
 * known once the kernel has counted (Sec. V-B enlarges FIFOs likewise).
 * Returns 0 for an unsupported dtype. */
uint64_t spccl_stream_bound(uint64_t n, int32_t dtype);

/* Workspace for messages of up to n elements: a 256-byte control block
 * (the sticky device status), one 64-bit look-back word per partition of
 * 16384 elements and one per 256 partitions, two tile indexes of COO operands
 * (one 64-bit word per 4096-element tile plus one, each), one worst-case slot
 * of compacted values per partition (n elements' worth) and one of 32-bit
 * indices (COO outputs).  spccl_workspace_min_bytes covers the first three
 * regions.  A reduce whose workspace holds them gives each COO operand a tile
 * index (the first entry of every tile, tagged with the call, built from J by
 * one extra pass) so its tiles find their entries without searching J; tiles
 * the index leaves out (long runs of empty tiles) and every tile of a reduce
 * with a smaller workspace (at least the control block, for a dense result)
 * search.  A Pici-producing call runs as one launch whose partitions find
 * their offsets from their predecessors' counts while holding their tiles
 * (every call on a workspace of only spccl_workspace_min_bytes, and sizes
 * within the limits of spccl_set_single_pass_limit), or as two passes that
 * never wait while holding input data (count and park values in the slots,
 * then add up the counts per chunk of partitions and move).  Outputs are
 * identical.  COO outputs always take two passes and need the full
 * workspace.
 * Zero-fill a workspace once before first use (or clear it with
 * spccl_workspace_init); look-back words are tagged with a per-launch epoch,
 * so it needs no clearing between calls.  One workspace must not be used by
 * two calls in flight at once. */
uint64_t spccl_workspace_bytes(uint64_t n, int32_t dtype);
uint64_t spccl_workspace_min_bytes(uint64_t n, int32_t dtype);

/* Zero-fill a workspace with a fill kernel on `stream` (no memset nodes). */
spccl_status_t spccl_workspace_init(void* ws, uint64_t ws_bytes, void* stream);

/* An upper bound, in partitions of 16384 elements, on the Pici outputs that a
 * call whose workspace holds the value slots writes in one launch (each
 * partition finds its offset from the counts of the partitions before it in
 * its chunk of 256 and the sums of the earlier chunks: Sec. III-B phase 2, the
 * global scan); larger outputs take the count and place passes.  Within the
 * bound the library's own limits apply: fp32 outputs of dense sources at
 * every size, bf16 ones up to 2048 partitions, Pici (+) Pici -> Pici up to
 * 1024 partitions and from 2048 on (a kernel with one partition per wave).  Default UINT32_MAX (the library's limits alone); 0 keeps every such
 * call on two passes.  The ring steps of the spccl_vr_* collectives follow the
 * same limits per rank's message; COO outputs always take two passes, and a
 * workspace of only spccl_workspace_min_bytes always one.  Process-wide (every device and
 * thread), takes effect for later calls; outputs are identical either way.
 * Returns the previous bound. */
uint32_t spccl_set_single_pass_limit(uint32_t max_partitions);

/* Exact byte size of a COO message with nnz nonzeros (Sec. II-B sizes: a
 * 32-bit index and a value per nonzero; plus header and pad).  0 for an
 * unsupported dtype. */
uint64_t spccl_coo_bytes(int32_t dtype, uint64_t nnz);

/* Worst-case size of an n-element message in format fmt, or of the dense
 * message if that is larger (a sender may always fall back to dense).  A
 * COO output needs this capacity (every element present: 48 + pad + n *
 * (4 + elem_size)).  0 for an unsupported dtype or format. */
uint64_t spccl_message_bound(uint64_t n, int32_t dtype, int32_t fmt);

/* ---- codec (Sec. III-B format, Alg. 1 compression, Sec. III-C) ----------- */

/* Compress dense[0..n) into a Pici message at `out` (capacity out_bytes >=
 * spccl_stream_bound(n, dtype)): bit vector B, tile prefix sums I and
 * compacted values A, ordered tile -> column -> row.  The input is read
 * once; partition offsets are found in the same launch (each partition adds
 * up its predecessors' counts in two levels) or by a count and a place pass
 * (see spccl_set_single_pass_limit).  nnz is in the written header. */
spccl_status_t spccl_compress(const void* dense, uint64_t n, int32_t dtype,
                              void* out, uint64_t out_bytes,
                              void* ws, uint64_t ws_bytes, void* stream);

/* Expand a message (PICI, COO or DENSE, read from its header) of capacity
 * in_bytes into all n elements of `dense` (absent elements become +0.0).  A
 * COO tile's entries are found by searching J; entries outside their tile,
 * at or past n, or not strictly increasing flag SPCCL_ERR_CORRUPT_STREAM and
 * their tile reads as empty. */
spccl_status_t spccl_decompress(const void* in, uint64_t in_bytes,
                                void* dense, uint64_t n, int32_t dtype,
                                void* ws, uint64_t ws_bytes, void* stream);

/* Compress dense[0..n) into a COO message at `out` (capacity out_bytes >=
 * spccl_message_bound(n, dtype, SPCCL_FMT_COO)): the flat index and the
 * value of every present element, by increasing index (Sec. II-B; the
 * paper's collectives use it beside Pici, Sec. IV-D).  Three passes (count
 * and park entries per 16384-element partition, scan the partition counts,
 * place); needs ws_bytes >= spccl_workspace_bytes(n, dtype), else
 * SPCCL_ERR_WORKSPACE. */
spccl_status_t spccl_compress_coo(const void* dense, uint64_t n, int32_t dtype,
                                  void* out, uint64_t out_bytes,
                                  void* ws, uint64_t ws_bytes, void* stream);

/* Wrap dense[0..n) as a DENSE message (header + the n values) at `out`
 * (capacity out_bytes >= 48 + n * elem_size).  Dense sends carry the same
 * header as sparse ones (Sec. V-B); nnz is recorded as "not computed". */
spccl_status_t spccl_encode_dense(const void* dense, uint64_t n, int32_t dtype,
                                  void* out, uint64_t out_bytes, void* stream);

/* ---- reduction with fill-in (Sec. IV-B) --------------------------------- */

/* out = a (+) b elementwise over n elements.  An absent element (all-zero
 * bits) is the identity; two present elements are added (fp32: IEEE add,
 * nearest-even; bf16: fp32 add rounded once to bfloat16, nearest-even).  A
 * result is present iff its bits are nonzero, so an exact cancellation drops
 * the element from a Pici or COO output.  In a ring step `a` is the received
 * (earlier) contribution; the operation is commutative bit for bit.
 * Supported operand kinds: a, b each ARRAY, STREAM/PICI, STREAM/COO or
 * STREAM/DENSE; out ARRAY, STREAM/PICI, STREAM/COO or STREAM/DENSE.  Pici
 * and COO do not meet in one call (a COO operand with a Pici operand or a
 * Pici output, or a Pici operand with a COO output: SPCCL_ERR_UNSUPPORTED).
 * out may alias a or b only when all three are ARRAYs (in-place
 * accumulation).  A PICI or DENSE STREAM output needs capacity >=
 * spccl_stream_bound(n, dtype), a COO one spccl_message_bound(n, dtype,
 * SPCCL_FMT_COO) and the full workspace. */
spccl_status_t spccl_reduce(spccl_operand_t a, spccl_operand_t b, spccl_operand_t out,
                            uint64_t n, int32_t dtype,
                            void* ws, uint64_t ws_bytes, void* stream);

/* ---- all-gather receive side (Sec. IV-B) --------------------------------- */

/* dense_out[q*n_per_part .. (q+1)*n_per_part) = expand(parts[q]) for q < P.
 * parts (host array of P operands) are ARRAYs or STREAMs of any format
 * (a STREAM's format is read from its header; its fmt field is ignored).
 * Any P: parts are expanded 64 per launch, and every part is checked (kind,
 * alignment, capacity, no overlap with dense_out) before the first launch,
 * so a host-detectable error in any part leaves dense_out untouched. */
spccl_status_t spccl_gather_expand(const spccl_operand_t* parts, int32_t P,
                                   uint64_t n_per_part, int32_t dtype,
                                   void* dense_out, uint64_t out_bytes,
                                   void* ws, uint64_t ws_bytes, void* stream);

/* ---- sliced streams (Sec. III-B phase 2; Sec. V-B) -------------------------
 * Inside its collectives the paper compresses independent segments, one per
 * block, with block-local prefix sums, and sends every slice as its own
 * message behind its own header, in FIFO reservations sized for the worst
 * case.  A sliced stream is that layout for an n-element array: slot q, at
 * byte q * spccl_slice_bytes(dtype) of the buffer, holds elements
 * [SPCCL_SLICE_ELEMS q, min(n, SPCCL_SLICE_ELEMS (q + 1))) as an ordinary
 * message (Pici or dense only; the header layout above, n = the slice
 * length).
 * One device pass produces a slice, with no device-wide scan, and the
 * format of every slice is decided on the device: a produced slice is dense
 * iff its own sparsity (zeros / length, in double) is <= dense_thresh (give
 * a negative threshold to keep every slice in Pici).  Bytes of a slot past
 * its message are not written.  Sliced streams are 16-byte aligned and hold
 * spccl_slice_count(n) slots; dense arrays are element-aligned.  ws needs
 * only the control block (>= 256 bytes).  A slice of an input stream whose
 * header fails its checks sets SPCCL_ERR_CORRUPT_STREAM and its output
 * slice (or elements) is not written. */
#define SPCCL_SLICE_ELEMS 16384

uint64_t spccl_slice_count(uint64_t n);      /* ceil(n / SPCCL_SLICE_ELEMS) */
uint64_t spccl_slice_bytes(int32_t dtype);   /* bytes of one slot: the worst-case message of a full slice; 0 for an unsupported dtype */

/* dense[0..n) -> sliced stream at out (out_bytes >= slice_count * slice_bytes). */
spccl_status_t spccl_compress_sliced(const void* dense, uint64_t n, int32_t dtype, double dense_thresh,
                                     void* out, uint64_t out_bytes, void* ws, uint64_t ws_bytes, void* stream);

/* sliced stream at in -> all n elements of dense (absent elements +0.0). */
spccl_status_t spccl_decompress_sliced(const void* in, uint64_t in_bytes, void* dense, uint64_t n, int32_t dtype,
                                       void* ws, uint64_t ws_bytes, void* stream);

/* out = a (+) b (Sec. IV-B) with a a dense array and b a sliced stream; out
 * is a sliced stream (out_sliced != 0, formats by dense_thresh) or a dense
 * array, which may be a itself (in-place accumulation; no other overlap).
 * The reduce-scatter step of the paper's in-collective mode. */
spccl_status_t spccl_reduce_sliced(const void* a, const void* b, uint64_t b_bytes, void* out, uint64_t out_bytes,
                                   int32_t out_sliced, double dense_thresh, uint64_t n, int32_t dtype,
                                   void* ws, uint64_t ws_bytes, void* stream);

/* The virtual-rank send of a sliced stream: every slot's header.total_bytes,
 * read on the device (no host synchronisation). */
spccl_status_t spccl_copy_sliced(const void* src, uint64_t src_bytes, void* dst, uint64_t dst_bytes, uint64_t n,
                                 int32_t dtype, void* ws, uint64_t ws_bytes, void* stream);

/* Per-slice format tracking (Sec. IV-C applied per slice, as the paper's
 * in-collective decisions are made per slice, Sec. V-B): a tracker holds,
 * for each slice of an n-element array, sigma0 and the tracked sparsity
 * sigma_prev as two doubles (16 bytes per slice, 8-byte aligned device
 * memory, caller-owned).  The decisions are made on the device, so a ring
 * of tracked calls needs no host synchronisation between steps. */
uint64_t spccl_slice_tracker_bytes(uint64_t n);   /* 16 * spccl_slice_count(n) */

/* First send of a ring: compress dense[0..n) into a sliced stream; each
 * slice's measured sparsity becomes its sigma0 and sigma_prev, and the slice
 * is dense iff that sparsity <= tau.  fmt_out (device, optional) gets one
 * byte per slice: the format produced. */
spccl_status_t spccl_compress_sliced_tracked(const void* dense, uint64_t n, int32_t dtype, double tau,
                                             void* out, uint64_t out_bytes, double* tracker,
                                             uint64_t tracker_bytes, uint8_t* fmt_out,
                                             void* ws, uint64_t ws_bytes, void* stream);

/* A later send: out = a (+) b (dense array, sliced stream) as a sliced
 * stream; per slice, est = sigma_prev * sigma0 (Eq. 7): the slice is dense
 * iff est <= tau (sigma_prev := est), otherwise Pici (sigma_prev := its
 * measured sparsity).  No operand may overlap another. */
spccl_status_t spccl_reduce_sliced_tracked(const void* a, const void* b, uint64_t b_bytes, void* out,
                                           uint64_t out_bytes, double tau, double* tracker,
                                           uint64_t tracker_bytes, uint8_t* fmt_out, uint64_t n,
                                           int32_t dtype, void* ws, uint64_t ws_bytes, void* stream);

/* ---- compression without a caller workspace --------------------------------
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * message as spccl_compress, made by the one-launch kernels, whose scratch
 * (a status word, one look-back word per 16384-element partition and one per
 * 256 partitions) lives in a static device array of the library -- 128.5 KiB
 * plus a 256-byte control block, one copy per GPU, held until the process
 * ends.  The call allocates
 * nothing.  n <= SPCCL_STATIC_MAX_ELEMS, else SPCCL_ERR_UNSUPPORTED; other
 * argument errors as spccl_compress (out_bytes >= spccl_stream_bound).  Every
 * call on a GPU shares that GPU's array, so calls that overlap on one GPU
 * (two streams at once) race and must not be issued; calls in order on
 * streams are fine.  A device-side wait that exceeds its spin limit clears
 * the output header's magic, so the message is rejected as corrupt by every
 * reader. */
#define SPCCL_STATIC_MAX_ELEMS (1ull << 28)
spccl_status_t spccl_compress_static(const void* dense, uint64_t n, int32_t dtype, void* out, uint64_t out_bytes,
                                     void* stream);

/* ---- message transport and inspection ------------------------------------ */

/* The virtual-rank "send": copy header.total_bytes bytes of the message at
 * src (capacity src_bytes) to dst (capacity dst_bytes).  The size is read on
 * the device, so no host synchronisation is needed.  A message that does not
 * fit sets SPCCL_ERR_CORRUPT_STREAM in ws and copies nothing. */
spccl_status_t spccl_copy_message(const void* src, uint64_t src_bytes, void* dst, uint64_t dst_bytes,
                                  void* ws, uint64_t ws_bytes, void* stream);

/* Copy the 48-byte header of a device message to host_out (synchronizes). */
spccl_status_t spccl_read_header(const void* msg, spccl_header_t* host_out, void* stream);

/* Synchronize `stream`, return the sticky device status in ws and, if clear
 * != 0, reset it to SPCCL_OK. */
spccl_status_t spccl_read_status(void* ws, int32_t clear, void* stream);

const char* spccl_status_string(spccl_status_t s);

/* ---- ring collectives over P virtual ranks on one GPU (Sec. IV) ----------- */

/* Adaptive format policy (Sec. IV-C).  Defaults for Pici with fp32:
 * intra 0.6, inter 0.5, ag 0.1; the paper's COO values (Sec. IV-D) are
 * intra 0.8, inter 0.7, ag 0.5. */
typedef struct {
    double intra_thresh;     /* dense iff sparsity <= this on an intra-node link */
    double inter_thresh;     /* ... on an inter-node link */
    double ag_thresh;        /* all-reduce: gather densely iff estimate <= this */
    int32_t ranks_per_node;  /* link r -> r+1 is inter-node iff (r+1) % ranks_per_node == 0
                                and ranks_per_node < P; 0 = all links intra-node */
    int32_t adaptive;        /* 0: always sparse; 1: threshold rule; 2: always dense */
    int32_t sparse_fmt;      /* format of the sparse sends: SPCCL_FMT_PICI or SPCCL_FMT_COO */
} spccl_policy_t;

/* One send decision of one rank (host array; see spccl_vr_*). */
typedef struct {
    int32_t step, rank;
    int32_t fmt;             /* format of the message sent at this step */
    int32_t measured;        /* 1 if this step counted the nonzeros */
    uint64_t bytes;          /* message bytes, header included */
    uint64_t nnz;            /* counted nonzeros, or SPCCL_NNZ_UNKNOWN */
    double sigma;            /* tracked sparsity after this step (Eq. 7 estimate
                                or measurement); for an all-gather entry of an
                                all-reduce, the transition estimate */
} spccl_trace_t;

/* Scratch bytes the collectives need: P ranks exchanging messages of up to
 * msg_elems elements (n / P for reduce-scatter and all-reduce, n for
 * all-gather).  Holds one workspace and 3*P message buffers of the larger
 * of spccl_message_bound(msg_elems, dtype, SPCCL_FMT_COO) and
 * spccl_stream_bound(msg_elems, dtype) bytes (any format fits; for short
 * messages the Pici bound is the larger). */
uint64_t spccl_vr_scratch_bytes(int32_t P, uint64_t msg_elems, int32_t dtype);

/* Ring reduce-scatter (Sec. IV-B).  send: host array of P device pointers to
 * n-element inputs; recv: host array of P device pointers, rank r receives
 * the n/P-element chunk r: (((X_{r+1} (+) X_{r+2}) (+) ...) (+) X_{r-1}) (+) X_r.
 * At step s rank r sends chunk (r-s-1) mod P to rank r+1; step 0 compresses
 * and measures sigma0; later steps extrapolate sigma_prev * sigma0 (Eq. 7)
 * and send dense iff the estimate <= the link's threshold.  trace (host,
 * optional) gets P*(P-1) entries, step-major.  n % P == 0.  Buffers: no
 * recv[r] may overlap another rank's recv, any other rank's send or the
 * scratch, and recv[r] may lie in send[r] only as its own chunk r (in place,
 * recv[r] == send[r] + r * n/P elements); no send may overlap the scratch.
 * Any other overlap returns SPCCL_ERR_INVALID_ARG before anything is
 * launched. */
spccl_status_t spccl_vr_reduce_scatter(void* const* send, void* const* recv, int32_t P, uint64_t n,
                                       int32_t dtype, const spccl_policy_t* policy,
                                       void* scratch, uint64_t scratch_bytes,
                                       spccl_trace_t* trace, void* stream);

/* Ring all-gather (Sec. IV-B): each rank compresses its n-element part once
 * (in policy->sparse_fmt; NULL policy = Pici), the message travels the ring
 * unchanged, and every rank expands all P parts into recv[r] (P*n
 * elements).  Never switches to dense.  trace gets P entries.  Buffers: no
 * recv[r] may overlap another rank's recv, any other rank's send or the
 * scratch, and send[r] may lie in recv[r] only at its own place (send[r] ==
 * recv[r] + r * n elements); otherwise SPCCL_ERR_INVALID_ARG, before any
 * launch. */
spccl_status_t spccl_vr_all_gather(void* const* send, void* const* recv, int32_t P, uint64_t n,
                                   int32_t dtype, const spccl_policy_t* policy,
                                   void* scratch, uint64_t scratch_bytes,
                                   spccl_trace_t* trace, void* stream);

/* Ring all-reduce = reduce-scatter, then all-gather of the reduced chunks;
 * at the transition each rank gathers densely iff sigma_prev * sigma0 <=
 * ag_thresh (phase-aware switch, Sec. IV-C).  recv[r] gets n elements.
 * trace gets P*(P-1) + P entries.  No recv[r] may overlap any send, another
 * recv or the scratch (SPCCL_ERR_INVALID_ARG, before any launch). */
spccl_status_t spccl_vr_all_reduce(void* const* send, void* const* recv, int32_t P, uint64_t n,
                                   int32_t dtype, const spccl_policy_t* policy,
                                   void* scratch, uint64_t scratch_bytes,
                                   spccl_trace_t* trace, void* stream);

/* Ring reduce-scatter over sliced streams with the decisions on the device
 * (the paper's in-collective mode, Sec. V-B, with Sec. IV-C per slice):
 * step 0 compresses as spccl_compress_sliced_tracked does, later steps send
 * as spccl_copy_sliced and reduce as spccl_reduce_sliced_tracked, the last
 * receive reduces into recv[r] (n/P elements, the same values as
 * spccl_vr_reduce_scatter).  The P ranks' kernels of one ring step are one
 * launch (up to 32 ranks each), so no recv[r] may overlap another rank's
 * recv, any send buffer or the scratch (SPCCL_ERR_INVALID_ARG).  tau per link as in
 * spccl_policy_t (adaptive 0: never dense, 2: always); sparse_fmt must be
 * SPCCL_FMT_PICI.  The stream is synchronised once, at the end.  fmt_trace
 * (host, optional) gets the format of every slice sent: (P-1) * P * S bytes,
 * index (step * P + rank) * S + slice, S = spccl_slice_count(n / P). */
/* Scratch of the sliced collectives (device, 16-byte aligned): msg_elems is
 * the elements of one rank's message -- n / P for the reduce-scatter and the
 * all-reduce, n for the all-gather.  0 for an invalid P or dtype. */
uint64_t spccl_vr_sliced_scratch_bytes(int32_t P, uint64_t msg_elems, int32_t dtype);
spccl_status_t spccl_vr_reduce_scatter_sliced(void* const* send, void* const* recv, int32_t P, uint64_t n,
                                              int32_t dtype, const spccl_policy_t* policy,
                                              void* scratch, uint64_t scratch_bytes,
                                              uint8_t* fmt_trace, void* stream);

/* Ring all-gather over sliced streams (Sec. IV-B with the Sec. V-B slice
 * layout): every rank encodes its n-element part send[r] once, every slice
 * Pici (a standalone all-gather never densifies), and the stream travels the
 * ring unchanged; recv[r] (P*n elements) gets part q at q*n on every rank,
 * the same values as spccl_vr_all_gather.  One launch per kernel and hop
 * for up to 32 ranks; no recv[r] may overlap another rank's recv or any send
 * (SPCCL_ERR_INVALID_ARG).  Scratch: spccl_vr_sliced_scratch_bytes(P, n,
 * dtype).  fmt_trace (host, optional) gets the P * S slice formats, index
 * rank * S + slice, S = spccl_slice_count(n).  Synchronises the stream once,
 * at the end; P = 1 copies. */
spccl_status_t spccl_vr_all_gather_sliced(void* const* send, void* const* recv, int32_t P, uint64_t n,
                                          int32_t dtype, void* scratch, uint64_t scratch_bytes,
                                          uint8_t* fmt_trace, void* stream);

/* Ring all-reduce over sliced streams: the sliced reduce-scatter (rank r's
 * reduced chunk lands at r*n/P of recv[r]), then the sliced all-gather of
 * the reduced chunks.  At the transition every slice extrapolates once more
 * from its tracker, est = sigma_prev * sigma0, and is gathered densely iff
 * est <= policy->ag_thresh (Sec. IV-C per slice; adaptive 0: never, 2:
 * always).  recv[r] gets n elements, the same values as spccl_vr_all_reduce.
 * Buffer rules as spccl_vr_reduce_scatter_sliced; scratch:
 * spccl_vr_sliced_scratch_bytes(P, n / P, dtype).  fmt_rs (host, optional):
 * the reduce-scatter's (P-1) * P * S slice formats as there; fmt_ag (host,
 * optional): the all-gather's P * S, index rank * S + slice, S =
 * spccl_slice_count(n / P).  P = 1 copies and writes no formats. */
spccl_status_t spccl_vr_all_reduce_sliced(void* const* send, void* const* recv, int32_t P, uint64_t n,
                                          int32_t dtype, const spccl_policy_t* policy,
                                          void* scratch, uint64_t scratch_bytes,
                                          uint8_t* fmt_rs, uint8_t* fmt_ag, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SPCCL_H */
