/*
 * pici_oracle.c -- plain, slow, single-threaded CPU oracle for the Pici
 * hot path of SpCCL (arXiv 2607.04676).  TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load this library.  The GPU path never links, includes or calls it, and it
 * shares no code, header, table or constant generator with the GPU path.
 *
 * What is defined here, each function citing the passage it follows:
 *   - the Pici encoding of a dense array      (Sec. III-B, Alg. 1)
 *   - the 48-byte message header              (Sec. V-B)
 *   - decompression                           (Sec. III-C, last paragraph)
 *   - the elementwise reduction with fill-in  (Sec. IV-B; Sec. I on fill-in)
 *   - ring reduce-scatter / all-gather / all-reduce over P virtual ranks
 *                                             (Sec. II-A Eq. 2, Sec. IV-A/B)
 *   - the adaptive dense switch with Eq. 7    (Sec. IV-C)
 *   - sliced streams: one message per slice, block-local prefix sums
 *                                             (Sec. III-B phase 2, Sec. V-B)
 *   - the flat COO format (one 32-bit index and one value per nonzero) and
 *     its use in the same collectives            (Sec. II-B, Sec. IV-D)
 *
 * Pici is an exact encoding, so compression is written as its definition:
 * loops over tiles, columns and rows in the order the format fixes.  No
 * blocking, fusion or reordering.  Readings of points the paper leaves open
 * (bit order, index width, partial last tile, header layout, cancellation,
 * decision timing) are listed in the design notes and restated where used.
 *
 * Build: gcc -O2 -std=c99 -fPIC -shared (no fast-math: IEEE round-to-nearest,
 * denormals kept).
 */
#define _POSIX_C_SOURCE 199309L     /* clock_gettime, for the timing helper at the end */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#include <time.h>

/* ---- constants of the format (Sec. III-B) ---------------------------- */
#define ORC_TILE_ROWS 64u           /* a tile is 64 x 64 elements, row-major */
#define ORC_TILE_COLS 64u
#define ORC_TILE_ELEMS 4096u        /* k = 4096 bits of B per tile           */
#define ORC_HEADER_BYTES 48u        /* message header size (Sec. V-B)        */
#define ORC_MAGIC 0x49434950u       /* bytes 'P','I','C','I'                 */
#define ORC_NNZ_UNKNOWN UINT64_MAX  /* dense message: nnz not computed      */

/* dtype codes and format / kind codes of the library interface */
enum { ORC_F32 = 0, ORC_BF16 = 1 };
enum { ORC_FMT_DENSE = 0, ORC_FMT_PICI = 1, ORC_FMT_COO = 2 };
enum { ORC_ARRAY = 0, ORC_STREAM = 1 };
/* status codes of the library interface */
enum { ORC_OK = 0, ORC_ERR_INVALID_ARG = 1, ORC_ERR_CAPACITY = 2,
       ORC_ERR_UNSUPPORTED = 3, ORC_ERR_CORRUPT_STREAM = 4 };

static uint64_t elem_size(int dtype) { return dtype == ORC_BF16 ? 2u : 4u; }

/* number of 64x64 tiles covering n elements: T = ceil(n / 4096) */
uint64_t orc_num_tiles(uint64_t n) { return (n + ORC_TILE_ELEMS - 1) / ORC_TILE_ELEMS; }

static uint64_t align16(uint64_t x) { return (x + 15u) / 16u * 16u; }

/* Byte offsets of a Pici message: header, then B (one 64-bit word per tile
 * column, 64 per tile), then I (T+1 unsigned 32-bit prefix sums), zero pad to
 * a 16-byte boundary, then A (nnz values).  Sec. III-B gives the components
 * and their sizes; Sec. V-B says a header precedes every message. */
uint64_t orc_off_I(uint64_t n) { return ORC_HEADER_BYTES + 512u * orc_num_tiles(n); }
uint64_t orc_off_A(uint64_t n) { return align16(orc_off_I(n) + 4u * (orc_num_tiles(n) + 1u)); }
uint64_t orc_pici_bytes(uint64_t n, int dtype, uint64_t nnz) {
    return orc_off_A(n) + nnz * elem_size(dtype);
}
uint64_t orc_dense_bytes(uint64_t n, int dtype) { return ORC_HEADER_BYTES + n * elem_size(dtype); }
/* worst-case message size: a Pici message with every element present
 * (Sec. V-B enlarges the FIFOs so that the worst case fits). */
uint64_t orc_stream_bound(uint64_t n, int dtype) {
    uint64_t p = orc_pici_bytes(n, dtype, n), d = orc_dense_bytes(n, dtype);
    return p > d ? p : d;
}

/* A COO message (Sec. II-B: the one-dimensional variant, a single flat
 * 32-bit index per nonzero, and its value): the header, then J (nnz unsigned
 * 32-bit indices, strictly increasing), zero pad to a 16-byte boundary, then
 * V (the nnz values, in index order).  The paper sizes COO as 32-bit indices
 * plus 32-bit values; the layout (indices apart from values) is this
 * library's. */
uint64_t orc_coo_off_V(uint64_t nnz) { return align16(ORC_HEADER_BYTES + 4u * nnz); }
uint64_t orc_coo_bytes(int dtype, uint64_t nnz) { return orc_coo_off_V(nnz) + nnz * elem_size(dtype); }
/* worst case of any message of n elements in format fmt (the dense message
 * included: a sender may always fall back to it) */
uint64_t orc_message_bound(uint64_t n, int dtype, int fmt) {
    uint64_t d = orc_dense_bytes(n, dtype);
    uint64_t w = fmt == ORC_FMT_COO ? orc_coo_bytes(dtype, n) : (fmt == ORC_FMT_PICI ? orc_pici_bytes(n, dtype, n) : d);
    return w > d ? w : d;
}

/* ---- little-endian field access, byte by byte ------------------------- */
static void put_u16(uint8_t* p, uint16_t v) { p[0] = (uint8_t)v; p[1] = (uint8_t)(v >> 8); }
static void put_u32(uint8_t* p, uint32_t v) { for (int i = 0; i < 4; i++) p[i] = (uint8_t)(v >> (8 * i)); }
static void put_u64(uint8_t* p, uint64_t v) { for (int i = 0; i < 8; i++) p[i] = (uint8_t)(v >> (8 * i)); }
static uint16_t get_u16(const uint8_t* p) { return (uint16_t)(p[0] | (p[1] << 8)); }
static uint32_t get_u32(const uint8_t* p) {
    uint32_t v = 0; for (int i = 3; i >= 0; i--) v = (v << 8) | p[i]; return v;
}
static uint64_t get_u64(const uint8_t* p) {
    uint64_t v = 0; for (int i = 7; i >= 0; i--) v = (v << 8) | p[i]; return v;
}

/* element i of a dense array as its raw bit pattern */
static uint32_t load_bits(const void* d, int dtype, uint64_t i) {
    if (dtype == ORC_BF16) { uint16_t v; memcpy(&v, (const uint8_t*)d + 2 * i, 2); return v; }
    uint32_t v; memcpy(&v, (const uint8_t*)d + 4 * i, 4); return v;
}
static void store_bits(void* d, int dtype, uint64_t i, uint32_t v) {
    if (dtype == ORC_BF16) { uint16_t w = (uint16_t)v; memcpy((uint8_t*)d + 2 * i, &w, 2); return; }
    memcpy((uint8_t*)d + 4 * i, &v, 4);
}

/* An element is "nonzero" (present) iff its raw bit pattern is not all zero
 * bits.  Sec. III-B speaks of zero and nonzero elements; reading the raw
 * pattern keeps -0.0 so that decompress(compress(x)) is x bit for bit. */
static int present(uint32_t bits) { return bits != 0; }

static int popcount64(uint64_t w) {
    int c = 0;
    for (int b = 0; b < 64; b++) c += (int)((w >> b) & 1u);
    return c;
}

static void write_header(uint8_t* s, int fmt, int dtype, uint64_t n, uint64_t nnz,
                         uint64_t off_I, uint64_t off_A, uint64_t total) {
    memset(s, 0, ORC_HEADER_BYTES);
    put_u32(s + 0, ORC_MAGIC);
    put_u16(s + 4, (uint16_t)fmt);
    put_u16(s + 6, (uint16_t)dtype);
    put_u64(s + 8, n);
    put_u64(s + 16, nnz);
    put_u64(s + 24, off_I);
    put_u64(s + 32, off_A);
    put_u64(s + 40, total);
}

/* ---- Pici compression (Sec. III-B and Alg. 1) ------------------------- */
/* Encodes dense[0..n) as a Pici message into stream (capacity cap bytes).
 * B[64t + c] bit r is set iff element 4096t + 64r + c exists (< n) and is
 * present (the tile is row-major, each B word is one tile column, the least
 * significant bit is row 0).  I[t] is the exclusive prefix sum of the tile
 * nonzero counts and I[T] = nnz.  A holds the present values ordered by
 * tile, then column, then row.  Returns a status; *nnz_out gets nnz. */
int orc_compress(const void* dense, uint64_t n, int dtype, uint8_t* stream, uint64_t cap,
                 uint64_t* nnz_out) {
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_ERR_UNSUPPORTED;
    if (n >= ((uint64_t)1 << 32)) return ORC_ERR_UNSUPPORTED;   /* I is 32-bit */
    const uint64_t T = orc_num_tiles(n);
    const uint64_t offI = orc_off_I(n), offA = orc_off_A(n);
    if (cap < offA) return ORC_ERR_CAPACITY;

    /* Phase 1: bit vector B, one 64-bit word per tile column */
    uint64_t* B = (uint64_t*)calloc(T * 64 + 1, sizeof(uint64_t));
    if (!B) return ORC_ERR_INVALID_ARG;
    for (uint64_t t = 0; t < T; t++)
        for (uint64_t c = 0; c < ORC_TILE_COLS; c++) {
            uint64_t w = 0;
            for (uint64_t r = 0; r < ORC_TILE_ROWS; r++) {
                uint64_t i = ORC_TILE_ELEMS * t + ORC_TILE_COLS * r + c;
                if (i < n && present(load_bits(dense, dtype, i))) w |= (uint64_t)1 << r;
            }
            B[64 * t + c] = w;
        }
    /* Phase 2: exclusive prefix sum of tile counts; I[T] = nnz */
    uint64_t* I = (uint64_t*)calloc(T + 1, sizeof(uint64_t));
    if (!I) { free(B); return ORC_ERR_INVALID_ARG; }
    I[0] = 0;
    for (uint64_t t = 0; t < T; t++) {
        uint64_t cnt = 0;
        for (uint64_t c = 0; c < 64; c++) cnt += (uint64_t)popcount64(B[64 * t + c]);
        I[t + 1] = I[t] + cnt;
    }
    const uint64_t nnz = I[T];
    const uint64_t total = offA + nnz * elem_size(dtype);
    if (cap < total) { free(B); free(I); return ORC_ERR_CAPACITY; }

    memset(stream, 0, offA);
    write_header(stream, ORC_FMT_PICI, dtype, n, nnz, offI, offA, total);
    for (uint64_t j = 0; j < 64 * T; j++) put_u64(stream + ORC_HEADER_BYTES + 8 * j, B[j]);
    for (uint64_t t = 0; t <= T; t++) put_u32(stream + offI + 4 * t, (uint32_t)I[t]);

    /* Phase 3: compact present values into A, tile -> column -> row */
    uint8_t* A = stream + offA;
    uint64_t k = 0;
    for (uint64_t t = 0; t < T; t++)
        for (uint64_t c = 0; c < 64; c++)
            for (uint64_t r = 0; r < 64; r++)
                if ((B[64 * t + c] >> r) & 1u) {
                    uint64_t i = ORC_TILE_ELEMS * t + ORC_TILE_COLS * r + c;
                    store_bits(A, dtype, k, load_bits(dense, dtype, i));
                    k++;
                }
    free(B); free(I);
    if (k != nnz) return ORC_ERR_CORRUPT_STREAM;   /* cannot happen */
    if (nnz_out) *nnz_out = nnz;
    return ORC_OK;
}

/* A dense message: the header (format DENSE, nnz not computed) followed by
 * the n values (Sec. V-B: every message carries the header). */
int orc_encode_dense(const void* dense, uint64_t n, int dtype, uint8_t* stream, uint64_t cap) {
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_ERR_UNSUPPORTED;
    uint64_t total = orc_dense_bytes(n, dtype);
    if (cap < total) return ORC_ERR_CAPACITY;
    write_header(stream, ORC_FMT_DENSE, dtype, n, ORC_NNZ_UNKNOWN, 0, ORC_HEADER_BYTES, total);
    memcpy(stream + ORC_HEADER_BYTES, dense, n * elem_size(dtype));
    return ORC_OK;
}

/* ---- COO compression (Sec. II-B; used as in Sec. IV-D) ---------------- */
/* Encodes dense[0..n) as a COO message: every present element, in index
 * order, contributes its flat index to J and its value to V. */
int orc_compress_coo(const void* dense, uint64_t n, int dtype, uint8_t* stream, uint64_t cap,
                     uint64_t* nnz_out) {
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_ERR_UNSUPPORTED;
    if (n >= ((uint64_t)1 << 32)) return ORC_ERR_UNSUPPORTED;   /* 32-bit indices */
    uint64_t nnz = 0;
    for (uint64_t i = 0; i < n; i++) nnz += present(load_bits(dense, dtype, i)) ? 1u : 0u;
    const uint64_t offV = orc_coo_off_V(nnz), total = orc_coo_bytes(dtype, nnz);
    if (cap < total) return ORC_ERR_CAPACITY;
    memset(stream, 0, offV);
    write_header(stream, ORC_FMT_COO, dtype, n, nnz, ORC_HEADER_BYTES, offV, total);
    uint64_t k = 0;
    for (uint64_t i = 0; i < n; i++) {
        uint32_t v = load_bits(dense, dtype, i);
        if (!present(v)) continue;
        put_u32(stream + ORC_HEADER_BYTES + 4 * k, (uint32_t)i);
        store_bits(stream + offV, dtype, k, v);
        k++;
    }
    if (nnz_out) *nnz_out = nnz;
    return ORC_OK;
}

/* Header and index checks of a message of capacity cap that should hold n
 * elements of dtype.  Returns ORC_OK or ORC_ERR_CORRUPT_STREAM. */
int orc_validate(const uint8_t* s, uint64_t cap, uint64_t n, int dtype) {
    if (cap < ORC_HEADER_BYTES) return ORC_ERR_CORRUPT_STREAM;
    if (get_u32(s) != ORC_MAGIC) return ORC_ERR_CORRUPT_STREAM;
    int fmt = get_u16(s + 4), dt = get_u16(s + 6);
    uint64_t hn = get_u64(s + 8), nnz = get_u64(s + 16), offI = get_u64(s + 24),
             offA = get_u64(s + 32), total = get_u64(s + 40);
    if (dt != dtype || hn != n || total > cap) return ORC_ERR_CORRUPT_STREAM;
    if (fmt == ORC_FMT_DENSE) {
        if (offA != ORC_HEADER_BYTES || total != orc_dense_bytes(n, dtype)) return ORC_ERR_CORRUPT_STREAM;
        return ORC_OK;
    }
    if (fmt == ORC_FMT_COO) {
        if (nnz > n || offI != ORC_HEADER_BYTES || offA != orc_coo_off_V(nnz) ||
            total != orc_coo_bytes(dtype, nnz))
            return ORC_ERR_CORRUPT_STREAM;
        /* indices strictly increasing and inside the array */
        for (uint64_t k = 0; k < nnz; k++) {
            uint64_t j = get_u32(s + offI + 4 * k);
            if (j >= n) return ORC_ERR_CORRUPT_STREAM;
            if (k > 0 && j <= (uint64_t)get_u32(s + offI + 4 * (k - 1))) return ORC_ERR_CORRUPT_STREAM;
        }
        return ORC_OK;
    }
    if (fmt != ORC_FMT_PICI) return ORC_ERR_CORRUPT_STREAM;
    if (offI != orc_off_I(n) || offA != orc_off_A(n) || nnz > n ||
        total != orc_pici_bytes(n, dtype, nnz))
        return ORC_ERR_CORRUPT_STREAM;
    const uint64_t T = orc_num_tiles(n);
    if (get_u32(s + offI) != 0) return ORC_ERR_CORRUPT_STREAM;
    for (uint64_t t = 0; t < T; t++) {
        uint64_t cnt = 0;
        for (uint64_t c = 0; c < 64; c++)
            cnt += (uint64_t)popcount64(get_u64(s + ORC_HEADER_BYTES + 8 * (64 * t + c)));
        if ((uint64_t)get_u32(s + offI + 4 * (t + 1)) != (uint64_t)get_u32(s + offI + 4 * t) + cnt)
            return ORC_ERR_CORRUPT_STREAM;
    }
    if ((uint64_t)get_u32(s + offI + 4 * T) != nnz) return ORC_ERR_CORRUPT_STREAM;
    return ORC_OK;
}

/* ---- decompression (Sec. III-C: the compaction phase run backwards) --- */
/* Writes all n elements of dense: absent elements become +0.0, present ones
 * take their value from A in tile -> column -> row order.  Accepts a Pici, a
 * COO or a dense message. */
int orc_decompress(const uint8_t* s, uint64_t cap, void* dense, uint64_t n, int dtype) {
    int st = orc_validate(s, cap, n, dtype);
    if (st != ORC_OK) return st;
    if (get_u16(s + 4) == ORC_FMT_DENSE) {
        memcpy(dense, s + ORC_HEADER_BYTES, n * elem_size(dtype));
        return ORC_OK;
    }
    if (get_u16(s + 4) == ORC_FMT_COO) {   /* read the index-value pairs back (Sec. IV-D) */
        const uint64_t nnz = get_u64(s + 16), offV = get_u64(s + 32);
        memset(dense, 0, n * elem_size(dtype));
        for (uint64_t k = 0; k < nnz; k++)
            store_bits(dense, dtype, get_u32(s + ORC_HEADER_BYTES + 4 * k), load_bits(s + offV, dtype, k));
        return ORC_OK;
    }
    const uint64_t T = orc_num_tiles(n);
    const uint8_t* A = s + get_u64(s + 32);
    memset(dense, 0, n * elem_size(dtype));
    uint64_t k = 0;
    for (uint64_t t = 0; t < T; t++)
        for (uint64_t c = 0; c < 64; c++) {
            uint64_t w = get_u64(s + ORC_HEADER_BYTES + 8 * (64 * t + c));
            for (uint64_t r = 0; r < 64; r++)
                if ((w >> r) & 1u) {
                    uint64_t i = ORC_TILE_ELEMS * t + ORC_TILE_COLS * r + c;
                    if (i >= n) return ORC_ERR_CORRUPT_STREAM;   /* bit beyond the array */
                    store_bits(dense, dtype, i, load_bits(A, dtype, k));
                    k++;
                }
        }
    return ORC_OK;
}

/* ---- elementwise reduction (Sec. IV-B; fill-in as in Sec. I) ----------- */
/* bfloat16 value of a finite double x, rounded to nearest with ties to even:
 * scale x by the spacing q of bfloat16 numbers at its magnitude (8 significant
 * bits for normal numbers, a fixed 2^-133 below 2^-126), round the scaled
 * value to an integer with ties to even, scale back.  Exact in double. */
static uint16_t bf16_from_double(double x) {
    if (x == 0.0) return signbit(x) ? 0x8000u : 0x0000u;
    int e;
    (void)frexp(x, &e);                 /* |x| = m * 2^e with 0.5 <= m < 1 */
    int qexp = e - 8;
    if (qexp < -133) qexp = -133;
    double q = ldexp(1.0, qexp);
    double r = nearbyint(x / q) * q;    /* default rounding: nearest, ties even */
    if (fabs(r) >= ldexp(1.0, 128)) return signbit(x) ? 0xFF80u : 0x7F80u;   /* overflow */
    float f = (float)r;                 /* exact: r has at most 8 significant bits */
    uint32_t u; memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}
static double double_of_bf16(uint16_t h) {
    uint32_t u = (uint32_t)h << 16; float f; memcpy(&f, &u, 4); return (double)f;
}

/* a (+) b on raw bit patterns: an absent operand (all-zero bits) is the
 * identity, so a single present operand passes through unchanged (this keeps
 * a lone -0.0); two present operands are added.  fp32: IEEE binary32 add,
 * round to nearest even.  bf16: the exactly rounded bfloat16 of the sum.
 * The result counts as present iff its bits are nonzero, so an exact
 * cancellation x + (-x) = +0.0 drops the element, as accumulating densely and
 * then compressing again does (Sec. IV-B). */
uint32_t orc_oplus(uint32_t a, uint32_t b, int dtype) {
    if (!present(b)) return a;
    if (!present(a)) return b;
    if (dtype == ORC_BF16)
        return bf16_from_double(double_of_bf16((uint16_t)a) + double_of_bf16((uint16_t)b));
    float fa, fb; memcpy(&fa, &a, 4); memcpy(&fb, &b, 4);
    volatile float fs = fa + fb;        /* one binary32 addition */
    float f = fs; uint32_t u; memcpy(&u, &f, 4);
    return u;
}

/* an operand of a reduction: a raw dense array of n elements, or a message */
static int decode_operand(int kind, const void* p, uint64_t cap, uint64_t n, int dtype, void* dense) {
    if (kind == ORC_ARRAY) { memcpy(dense, p, n * elem_size(dtype)); return ORC_OK; }
    if (kind == ORC_STREAM) return orc_decompress((const uint8_t*)p, cap, dense, n, dtype);
    return ORC_ERR_INVALID_ARG;
}

/* out = a (+) b over n elements.  Operands are dense arrays or messages of
 * any format; the output is a dense array, or a message in format
 * out_fmt.  Follows the paper's reduce step literally: accumulate densely,
 * then (for a Pici output) compress the dense result again. */
int orc_reduce(int kind_a, const void* a, uint64_t cap_a, int kind_b, const void* b, uint64_t cap_b,
               int kind_out, int out_fmt, void* out, uint64_t cap_out, uint64_t n, int dtype,
               uint64_t* nnz_out) {
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_ERR_UNSUPPORTED;
    const uint64_t s = elem_size(dtype);
    void* da = malloc(n * s + 1); void* db = malloc(n * s + 1); void* dr = malloc(n * s + 1);
    int st = ORC_ERR_INVALID_ARG;
    if (!da || !db || !dr) goto done;
    st = decode_operand(kind_a, a, cap_a, n, dtype, da); if (st) goto done;
    st = decode_operand(kind_b, b, cap_b, n, dtype, db); if (st) goto done;
    for (uint64_t i = 0; i < n; i++)
        store_bits(dr, dtype, i, orc_oplus(load_bits(da, dtype, i), load_bits(db, dtype, i), dtype));
    if (kind_out == ORC_ARRAY) { memcpy(out, dr, n * s); st = ORC_OK; }
    else if (out_fmt == ORC_FMT_PICI) st = orc_compress(dr, n, dtype, (uint8_t*)out, cap_out, nnz_out);
    else if (out_fmt == ORC_FMT_COO) st = orc_compress_coo(dr, n, dtype, (uint8_t*)out, cap_out, nnz_out);
    else if (out_fmt == ORC_FMT_DENSE) st = orc_encode_dense(dr, n, dtype, (uint8_t*)out, cap_out);
    else st = ORC_ERR_INVALID_ARG;
done:
    free(da); free(db); free(dr);
    return st;
}

/* ---- ring collectives over P virtual ranks (Sec. IV-A, IV-B, IV-C) ---- */
typedef struct {
    double intra_thresh;   /* 0.6 for Pici, fp32 reduce-scatter (Sec. IV-C) */
    double inter_thresh;   /* 0.5 */
    double ag_thresh;      /* 0.1, at the RS -> AG transition of all-reduce */
    int ranks_per_node;    /* link r -> r+1 is inter-node iff (r+1) % ranks_per_node == 0 */
    int adaptive;          /* 0: never switch to dense; 1: threshold rule; 2: always dense */
    int sparse_fmt;        /* format of the sparse sends: ORC_FMT_PICI, or ORC_FMT_COO (Sec. IV-D) */
} orc_policy_t;

typedef struct {
    int32_t step, rank;
    int32_t fmt;           /* format of the message rank sends at this step */
    int32_t measured;      /* 1 if this step computed the nonzero count */
    uint64_t bytes;        /* total message bytes, header included */
    uint64_t nnz;          /* counted nonzeros, or UINT64_MAX if not computed */
    double sigma;          /* tracked sparsity after this step's update */
} orc_trace_t;

static double tau_link(const orc_policy_t* pol, int r, int P) {
    int rpn = pol->ranks_per_node > 0 ? pol->ranks_per_node : P;
    return ((r + 1) % rpn == 0 && rpn < P) ? pol->inter_thresh : pol->intra_thresh;
}

/* sparsity of an m-element message with nnz nonzeros: (m - nnz) / m */
static double sparsity(uint64_t m, uint64_t nnz) {
    return m == 0 ? 1.0 : (double)(m - nnz) / (double)m;
}

/* the dense-send rule: send dense iff sparsity <= tau (inclusive) */
static int go_dense(const orc_policy_t* pol, double sigma, double tau) {
    if (pol->adaptive == 0) return 0;
    if (pol->adaptive == 2) return 1;
    return sigma <= tau;
}

static void put_trace(orc_trace_t* tr, int idx, int step, int rank, int fmt, int measured,
                      uint64_t bytes, uint64_t nnz, double sigma) {
    if (!tr) return;
    tr[idx].step = step; tr[idx].rank = rank; tr[idx].fmt = fmt; tr[idx].measured = measured;
    tr[idx].bytes = bytes; tr[idx].nnz = nnz; tr[idx].sigma = sigma;
}

static uint64_t msg_bytes(const uint8_t* s) { return get_u64(s + 40); }

/* the sparse encoding of a collective: Pici, or COO (Sec. IV-D) */
static int compress_fmt(int fmt, const void* dense, uint64_t n, int dtype, uint8_t* out, uint64_t cap,
                        uint64_t* nnz) {
    if (fmt == ORC_FMT_COO) return orc_compress_coo(dense, n, dtype, out, cap, nnz);
    if (fmt == ORC_FMT_PICI) return orc_compress(dense, n, dtype, out, cap, nnz);
    return ORC_ERR_INVALID_ARG;
}

/* Ring reduce-scatter.  send[r] holds rank r's n elements; recv[r] gets the
 * reduced chunk r (m = n / P elements).  At step s (0 <= s <= P-2) rank r
 * sends chunk (r - s - 1) mod P to rank r+1; the receiver folds in its own
 * contribution, received message first.  Rank j therefore ends with
 * (((X_{j+1} (+) X_{j+2}) (+) ...) (+) X_{j+P-1}) (+) X_j on chunk j.
 * Format choice per sending rank (Sec. IV-C):
 *   step 0:  compress, measure sigma0 = sigma_prev; dense iff sigma0 <= tau
 *   step s:  est = sigma_prev * sigma0 (Eq. 7); if est <= tau reduce to a
 *            dense message and track est, else reduce + compress and track
 *            the measured sparsity.
 * sigma_out[r] (optional) gets rank r's tracked sparsity after the last send
 * and sigma0_out[r] its sigma0.  trace gets P*(P-1) entries, step-major. */
int orc_ring_reduce_scatter(const void* const* send, void* const* recv, int P, uint64_t n, int dtype,
                            const orc_policy_t* pol, orc_trace_t* trace,
                            double* sigma0_out, double* sigma_out) {
    if (P < 1 || n % (uint64_t)P) return ORC_ERR_INVALID_ARG;
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_ERR_UNSUPPORTED;
    const uint64_t m = n / (uint64_t)P, s = elem_size(dtype);
    const int sfmt = pol->sparse_fmt;
    if (sfmt != ORC_FMT_PICI && sfmt != ORC_FMT_COO) return ORC_ERR_INVALID_ARG;
    const uint64_t cap = orc_message_bound(m, dtype, sfmt);
    int st = ORC_OK;
    if (P == 1) {
        memcpy(recv[0], send[0], m * s);
        if (sigma0_out) sigma0_out[0] = 1.0;
        if (sigma_out) sigma_out[0] = 1.0;
        return ORC_OK;
    }
    uint8_t** out_msg = (uint8_t**)calloc((size_t)P, sizeof(uint8_t*));
    uint8_t** in_msg = (uint8_t**)calloc((size_t)P, sizeof(uint8_t*));
    double* sig0 = (double*)calloc((size_t)P, sizeof(double));
    double* sigp = (double*)calloc((size_t)P, sizeof(double));
    uint8_t* tmp = (uint8_t*)malloc(cap);
    if (!out_msg || !in_msg || !sig0 || !sigp || !tmp) { st = ORC_ERR_INVALID_ARG; goto done; }
    for (int r = 0; r < P; r++) {
        out_msg[r] = (uint8_t*)malloc(cap); in_msg[r] = (uint8_t*)malloc(cap);
        if (!out_msg[r] || !in_msg[r]) { st = ORC_ERR_INVALID_ARG; goto done; }
    }
    /* step 0: every rank compresses the chunk it sends first */
    for (int r = 0; r < P; r++) {
        int c = (r - 1 + P) % P;
        const uint8_t* chunk = (const uint8_t*)send[r] + (uint64_t)c * m * s;
        uint64_t nnz = 0;
        st = compress_fmt(sfmt, chunk, m, dtype, tmp, cap, &nnz); if (st) goto done;
        sig0[r] = sigp[r] = sparsity(m, nnz);
        if (go_dense(pol, sig0[r], tau_link(pol, r, P))) {
            st = orc_encode_dense(chunk, m, dtype, out_msg[r], cap); if (st) goto done;
        } else {
            memcpy(out_msg[r], tmp, msg_bytes(tmp));
        }
        put_trace(trace, r, 0, r, (int)get_u16(out_msg[r] + 4), 1, msg_bytes(out_msg[r]), nnz, sigp[r]);
    }
    for (int step = 1; step <= P - 1; step++) {
        /* the sends of the previous step arrive: rank r gets rank r-1's message */
        for (int r = 0; r < P; r++) {
            const uint8_t* m_in = out_msg[(r - 1 + P) % P];
            memcpy(in_msg[r], m_in, msg_bytes(m_in));
        }
        for (int r = 0; r < P; r++) {
            int c = (r - step - 1 + 2 * P) % P;
            const uint8_t* own = (const uint8_t*)send[r] + (uint64_t)c * m * s;
            if (step == P - 1) {   /* last receive: chunk r, reduced into the output */
                st = orc_reduce(ORC_STREAM, in_msg[r], cap, ORC_ARRAY, own, 0, ORC_ARRAY, ORC_FMT_DENSE,
                                recv[r], 0, m, dtype, NULL);
                if (st) goto done;
                continue;
            }
            double est = sigp[r] * sig0[r];   /* Eq. 7 */
            int idx = step * P + r;
            if (go_dense(pol, est, tau_link(pol, r, P))) {
                st = orc_reduce(ORC_STREAM, in_msg[r], cap, ORC_ARRAY, own, 0, ORC_STREAM, ORC_FMT_DENSE,
                                out_msg[r], cap, m, dtype, NULL);
                if (st) goto done;
                sigp[r] = est;
                put_trace(trace, idx, step, r, ORC_FMT_DENSE, 0, msg_bytes(out_msg[r]), ORC_NNZ_UNKNOWN, sigp[r]);
            } else {
                uint64_t nnz = 0;
                st = orc_reduce(ORC_STREAM, in_msg[r], cap, ORC_ARRAY, own, 0, ORC_STREAM, sfmt,
                                out_msg[r], cap, m, dtype, &nnz);
                if (st) goto done;
                sigp[r] = sparsity(m, nnz);
                put_trace(trace, idx, step, r, sfmt, 1, msg_bytes(out_msg[r]), nnz, sigp[r]);
            }
        }
    }
    for (int r = 0; r < P; r++) {
        if (sigma0_out) sigma0_out[r] = sig0[r];
        if (sigma_out) sigma_out[r] = sigp[r];
    }
done:
    if (out_msg) for (int r = 0; r < P; r++) free(out_msg[r]);
    if (in_msg) for (int r = 0; r < P; r++) free(in_msg[r]);
    free(out_msg); free(in_msg); free(sig0); free(sigp); free(tmp);
    return st;
}

/* Ring all-gather over messages.  part[q] is the n-element dense
 * contribution of rank q; fmt[q] the format rank q sends it in.  Each rank
 * encodes its contribution once and the message is forwarded unchanged
 * around the ring (Sec. IV-B); every receiver expands each message into
 * out[r] + q*n.  A rank's own part is copied from its input.  trace gets P
 * entries (step = trace_step). */
static int ring_all_gather_fmt(const void* const* part, const int* fmt, void* const* out, int P, uint64_t n,
                               int dtype, orc_trace_t* trace, int trace_step, const double* sig_track) {
    /* a part goes out dense, Pici or COO: room for the largest of the three
     * (COO's bound is the larger one except for short parts) */
    const uint64_t s = elem_size(dtype), cp = orc_message_bound(n, dtype, ORC_FMT_PICI),
                   cc = orc_message_bound(n, dtype, ORC_FMT_COO), cap = cp > cc ? cp : cc;
    int st = ORC_OK;
    uint8_t** msg = (uint8_t**)calloc((size_t)P, sizeof(uint8_t*));
    uint8_t* hop = (uint8_t*)malloc(cap);
    if (!msg || !hop) { st = ORC_ERR_INVALID_ARG; goto done; }
    for (int q = 0; q < P; q++) {
        msg[q] = (uint8_t*)malloc(cap);
        if (!msg[q]) { st = ORC_ERR_INVALID_ARG; goto done; }
        uint64_t nnz = ORC_NNZ_UNKNOWN;
        if (fmt[q] == ORC_FMT_DENSE) st = orc_encode_dense(part[q], n, dtype, msg[q], cap);
        else st = compress_fmt(fmt[q], part[q], n, dtype, msg[q], cap, &nnz);
        if (st) goto done;
        double sig = sig_track ? sig_track[q] : sparsity(n, nnz);
        put_trace(trace, q, trace_step, q, fmt[q], fmt[q] != ORC_FMT_DENSE, msg_bytes(msg[q]), nnz, sig);
    }
    for (int r = 0; r < P; r++) {
        memcpy((uint8_t*)out[r] + (uint64_t)r * n * s, part[r], n * s);
        /* step k brings rank r the message of rank r-1-k, forwarded k times */
        for (int k = 0; k < P - 1; k++) {
            int q = ((r - 1 - k) % P + P) % P;
            memcpy(hop, msg[q], msg_bytes(msg[q]));
            st = orc_decompress(hop, cap, (uint8_t*)out[r] + (uint64_t)q * n * s, n, dtype);
            if (st) goto done;
        }
    }
done:
    if (msg) for (int q = 0; q < P; q++) free(msg[q]);
    free(msg); free(hop);
    return st;
}

/* Standalone all-gather in sparse format sparse_fmt (Pici or COO): never
 * switches to dense (it does not densify). */
int orc_ring_all_gather(const void* const* part, void* const* out, int P, uint64_t n, int dtype,
                        int sparse_fmt, orc_trace_t* trace) {
    if (P < 1) return ORC_ERR_INVALID_ARG;
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_ERR_UNSUPPORTED;
    if (sparse_fmt != ORC_FMT_PICI && sparse_fmt != ORC_FMT_COO) return ORC_ERR_INVALID_ARG;
    int* fmt = (int*)malloc(sizeof(int) * (size_t)P);
    if (!fmt) return ORC_ERR_INVALID_ARG;
    for (int q = 0; q < P; q++) fmt[q] = sparse_fmt;
    int st = ring_all_gather_fmt(part, fmt, out, P, n, dtype, trace, 0, NULL);
    free(fmt);
    return st;
}

/* All-reduce = ring reduce-scatter, then ring all-gather of the reduced
 * chunks (Sec. IV-B).  At the transition each rank extrapolates once more,
 * est = sigma_prev * sigma0, and gathers densely iff est <= ag_thresh
 * (phase-aware switch, Sec. IV-C).  out[r] gets n elements.  trace gets
 * P*(P-1) reduce-scatter entries followed by P all-gather entries (step P-1). */
int orc_ring_all_reduce(const void* const* send, void* const* out, int P, uint64_t n, int dtype,
                        const orc_policy_t* pol, orc_trace_t* trace) {
    if (P < 1 || n % (uint64_t)P) return ORC_ERR_INVALID_ARG;
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_ERR_UNSUPPORTED;
    const uint64_t m = n / (uint64_t)P, s = elem_size(dtype);
    int st = ORC_OK;
    void** red = (void**)calloc((size_t)P, sizeof(void*));
    double* sig0 = (double*)calloc((size_t)P, sizeof(double));
    double* sigp = (double*)calloc((size_t)P, sizeof(double));
    double* est = (double*)calloc((size_t)P, sizeof(double));
    int* fmt = (int*)calloc((size_t)P, sizeof(int));
    if (!red || !sig0 || !sigp || !est || !fmt) { st = ORC_ERR_INVALID_ARG; goto done; }
    for (int r = 0; r < P; r++) if (!(red[r] = malloc(m * s + 1))) { st = ORC_ERR_INVALID_ARG; goto done; }
    st = orc_ring_reduce_scatter(send, red, P, n, dtype, pol, trace, sig0, sigp);
    if (st) goto done;
    for (int r = 0; r < P; r++) {
        est[r] = sigp[r] * sig0[r];
        int dense = pol->adaptive == 2 ? 1 : (pol->adaptive == 0 ? 0 : est[r] <= pol->ag_thresh);
        fmt[r] = dense ? ORC_FMT_DENSE : pol->sparse_fmt;
    }
    st = ring_all_gather_fmt((const void* const*)red, fmt, out, P, m, dtype,
                             trace ? trace + (size_t)P * (size_t)(P - 1) : NULL, P - 1, est);
done:
    if (red) for (int r = 0; r < P; r++) free(red[r]);
    free(red); free(sig0); free(sigp); free(est); free(fmt);
    return st;
}

/* ---- sliced streams (Sec. III-B phase 2 and Sec. V-B) -------------------
 * Inside a collective the paper compresses independent segments, one per
 * block, each with a block-local prefix sum, and sends each slice as its own
 * message behind its own header, in FIFO reservations sized for the worst
 * case.  A sliced stream is that layout for a whole array: slice q holds the
 * ORC_SLICE_ELEMS consecutive elements starting at q * ORC_SLICE_ELEMS (the
 * last slice may be shorter) as an ordinary message -- Pici, or dense -- in
 * slot q of orc_slice_bytes(dtype) bytes.
 * Format of each slice: dense iff its own sparsity (counted zeros / length,
 * in double) is <= dense_thresh; a negative dense_thresh keeps every slice in
 * Pici.  (Reading: per slice, the count is part of producing the slice, so
 * the measured sparsity is used, not the Eq. 7 estimate.) */
#define ORC_SLICE_ELEMS 16384u

uint64_t orc_slice_count(uint64_t n) { return (n + ORC_SLICE_ELEMS - 1) / ORC_SLICE_ELEMS; }
uint64_t orc_slice_bytes(int dtype) { return orc_stream_bound(ORC_SLICE_ELEMS, dtype); }

static uint64_t slice_len(uint64_t n, uint64_t q) {
    const uint64_t lo = q * ORC_SLICE_ELEMS;
    return n - lo < ORC_SLICE_ELEMS ? n - lo : ORC_SLICE_ELEMS;
}

int orc_encode_sliced(const void* dense, uint64_t n, int dtype, double dense_thresh, uint8_t* out,
                      uint64_t cap) {
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_ERR_UNSUPPORTED;
    const uint64_t S = orc_slice_count(n), slot = orc_slice_bytes(dtype), s = elem_size(dtype);
    if (cap < S * slot) return ORC_ERR_CAPACITY;
    for (uint64_t q = 0; q < S; q++) {
        const uint64_t m = slice_len(n, q);
        const uint8_t* src = (const uint8_t*)dense + q * ORC_SLICE_ELEMS * s;
        uint64_t nnz = 0;
        for (uint64_t i = 0; i < m; i++) nnz += present(load_bits(src, dtype, i)) ? 1u : 0u;
        const double sigma = (double)(m - nnz) / (double)m;
        int st;
        if (sigma <= dense_thresh) {
            st = orc_encode_dense(src, m, dtype, out + q * slot, slot);
        } else {
            uint64_t got = 0;
            st = orc_compress(src, m, dtype, out + q * slot, slot, &got);
        }
        if (st != ORC_OK) return st;
    }
    return ORC_OK;
}

int orc_decode_sliced(const uint8_t* in, uint64_t cap, void* dense, uint64_t n, int dtype) {
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_ERR_UNSUPPORTED;
    const uint64_t S = orc_slice_count(n), slot = orc_slice_bytes(dtype), s = elem_size(dtype);
    if (cap < S * slot) return ORC_ERR_CAPACITY;
    for (uint64_t q = 0; q < S; q++) {
        /* a slot holds a Pici or a dense message; any other format is corrupt */
        if (get_u16(in + q * slot + 4) == ORC_FMT_COO) return ORC_ERR_CORRUPT_STREAM;
        int st = orc_decompress(in + q * slot, slot, (uint8_t*)dense + q * ORC_SLICE_ELEMS * s,
                                slice_len(n, q), dtype);
        if (st != ORC_OK) return st;
    }
    return ORC_OK;
}

/* out = a (+) b with a a dense array and b a sliced stream; the result is a
 * dense array (out_sliced = 0) or a sliced stream with the per-slice format
 * rule above.  Accumulate densely, then encode -- the paper's reduce step. */
int orc_reduce_sliced(const void* a, const uint8_t* b, uint64_t cap_b, int out_sliced, double dense_thresh,
                      void* out, uint64_t cap_out, uint64_t n, int dtype) {
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_ERR_UNSUPPORTED;
    const uint64_t s = elem_size(dtype);
    void* db = malloc(n * s + 1); void* dr = malloc(n * s + 1);
    int st = ORC_ERR_INVALID_ARG;
    if (!db || !dr) goto done;
    st = orc_decode_sliced(b, cap_b, db, n, dtype);
    if (st) goto done;
    for (uint64_t i = 0; i < n; i++)
        store_bits(dr, dtype, i, orc_oplus(load_bits(a, dtype, i), load_bits(db, dtype, i), dtype));
    if (!out_sliced) { memcpy(out, dr, n * s); st = ORC_OK; }
    else st = orc_encode_sliced(dr, n, dtype, dense_thresh, (uint8_t*)out, cap_out);
done:
    free(db); free(dr);
    return st;
}

/* ---- sliced ring reduce-scatter with per-slice decisions ---------------
 * The paper decides formats inside NCCLX per slice (Sec. V-B) with the
 * Sec. IV-C rule.  Reading: every slice q of the chunk a rank sends keeps its
 * own sigma0 (measured when the slice is first compressed, at step 0) and
 * its own tracked sparsity; at a later step the slice is sent dense iff
 * sigma_prev * sigma0 <= tau(link) (Eq. 7; the estimate is then tracked),
 * otherwise it is reduced and compressed and its measured sparsity is
 * tracked.  Step 0 sends a slice dense iff its sigma0 <= tau(link).  The last
 * receive reduces into the dense output.  Values are those of the plain ring
 * (formats never change values).  fmt_out (optional) gets the format of
 * every sent slice, indexed [(step * P + rank) * S + q], S = slices of a
 * chunk. */
static int rs_sliced(const void* const* send, void* const* recv, int P, uint64_t n, int dtype,
                     const orc_policy_t* pol, uint8_t* fmt_out, double* sig0_out, double* sigp_out);

int orc_ring_reduce_scatter_sliced(const void* const* send, void* const* recv, int P, uint64_t n, int dtype,
                                   const orc_policy_t* pol, uint8_t* fmt_out) {
    return rs_sliced(send, recv, P, n, dtype, pol, fmt_out, NULL, NULL);
}

/* The sliced ring reduce-scatter; sig0_out / sigp_out (optional, P * S
 * doubles each) get every rank's slice trackers as they stand after its last
 * tracked send (step P - 2). */
static int rs_sliced(const void* const* send, void* const* recv, int P, uint64_t n, int dtype,
                     const orc_policy_t* pol, uint8_t* fmt_out, double* sig0_out, double* sigp_out) {
    if (P < 1 || n % (uint64_t)P) return ORC_ERR_INVALID_ARG;
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_ERR_UNSUPPORTED;
    const uint64_t m = n / (uint64_t)P, s = elem_size(dtype);
    const uint64_t S = orc_slice_count(m), slot = orc_slice_bytes(dtype), cap = S * slot;
    int st = ORC_OK;
    if (P == 1) { memcpy(recv[0], send[0], m * s); return ORC_OK; }
    uint8_t** out_msg = (uint8_t**)calloc((size_t)P, sizeof(uint8_t*));
    uint8_t** in_msg = (uint8_t**)calloc((size_t)P, sizeof(uint8_t*));
    double* sig0 = (double*)calloc((size_t)(P * S + 1), sizeof(double));
    double* sigp = (double*)calloc((size_t)(P * S + 1), sizeof(double));
    uint8_t* acc = (uint8_t*)malloc(m * s + 1);
    uint8_t* tmp = (uint8_t*)malloc(slot + 1);
    if (!out_msg || !in_msg || !sig0 || !sigp || !acc || !tmp) { st = ORC_ERR_INVALID_ARG; goto done; }
    for (int r = 0; r < P; r++) {
        out_msg[r] = (uint8_t*)calloc(cap + 1, 1); in_msg[r] = (uint8_t*)calloc(cap + 1, 1);
        if (!out_msg[r] || !in_msg[r]) { st = ORC_ERR_INVALID_ARG; goto done; }
    }
    for (int step = 0; step <= P - 1; step++) {
        if (step > 0)   /* the sends of the previous step arrive: rank r gets rank r-1's stream */
            for (int r = 0; r < P; r++) memcpy(in_msg[r], out_msg[(r - 1 + P) % P], cap);
        for (int r = 0; r < P; r++) {
            int c = (r - step - 1 + 2 * P) % P;
            const uint8_t* own = (const uint8_t*)send[r] + (uint64_t)c * m * s;
            if (step == 0) {
                memcpy(acc, own, m * s);
            } else {
                st = orc_decode_sliced(in_msg[r], cap, acc, m, dtype); if (st) goto done;
                for (uint64_t i = 0; i < m; i++)
                    store_bits(acc, dtype, i, orc_oplus(load_bits(acc, dtype, i), load_bits(own, dtype, i), dtype));
            }
            if (step == P - 1) { memcpy(recv[r], acc, m * s); continue; }
            const double tau = tau_link(pol, r, P);
            for (uint64_t q = 0; q < S; q++) {
                const uint64_t len = slice_len(m, q);
                const uint8_t* src = acc + q * ORC_SLICE_ELEMS * s;
                uint64_t nnz = 0;
                for (uint64_t i = 0; i < len; i++) nnz += present(load_bits(src, dtype, i)) ? 1u : 0u;
                const double meas = (double)(len - nnz) / (double)len;
                double* s0 = &sig0[r * S + q]; double* sp = &sigp[r * S + q];
                int dense;
                if (step == 0) {
                    *s0 = *sp = meas;
                    dense = go_dense(pol, meas, tau);
                } else {
                    const double est = *sp * *s0;   /* Eq. 7 */
                    dense = go_dense(pol, est, tau);
                    *sp = dense ? est : meas;
                }
                uint8_t* dst = out_msg[r] + q * slot;
                if (dense) st = orc_encode_dense(src, len, dtype, dst, slot);
                else st = orc_compress(src, len, dtype, dst, slot, &nnz);
                if (st) goto done;
                if (fmt_out) fmt_out[((uint64_t)step * P + r) * S + q] = (uint8_t)(dense ? ORC_FMT_DENSE : ORC_FMT_PICI);
            }
        }
    }
    if (sig0_out) memcpy(sig0_out, sig0, sizeof(double) * (size_t)P * (size_t)S);
    if (sigp_out) memcpy(sigp_out, sigp, sizeof(double) * (size_t)P * (size_t)S);
done:
    if (out_msg) for (int r = 0; r < P; r++) free(out_msg[r]);
    if (in_msg) for (int r = 0; r < P; r++) free(in_msg[r]);
    free(out_msg); free(in_msg); free(sig0); free(sigp); free(acc); free(tmp);
    return st;
}

/* ---- sliced all-gather and all-reduce (Sec. IV-B over the Sec. V-B slice
 * layout) --------------------------------------------------------------
 * All-gather: every rank encodes its n-element part once as a sliced stream,
 * slice q of rank r in format fmt[r * S + q] (dense or Pici), the stream
 * travels the ring unchanged, and every rank decodes all P parts: out[r]
 * holds part q at q * n.  Decoding ignores the format, so the values are
 * those of the plain all-gather. */
static int ring_all_gather_sliced_fmt(const void* const* part, const uint8_t* fmt, void* const* out, int P,
                                      uint64_t n, int dtype) {
    const uint64_t s = elem_size(dtype), S = orc_slice_count(n), slot = orc_slice_bytes(dtype), cap = S * slot;
    int st = ORC_OK;
    uint8_t** msg = (uint8_t**)calloc((size_t)P, sizeof(uint8_t*));
    uint8_t* hop = (uint8_t*)malloc(cap + 1);
    if (!msg || !hop) { st = ORC_ERR_INVALID_ARG; goto done; }
    for (int q = 0; q < P; q++) {
        msg[q] = (uint8_t*)calloc(cap + 1, 1);
        if (!msg[q]) { st = ORC_ERR_INVALID_ARG; goto done; }
        for (uint64_t j = 0; j < S; j++) {
            const uint64_t len = slice_len(n, j);
            const uint8_t* src = (const uint8_t*)part[q] + j * ORC_SLICE_ELEMS * s;
            uint64_t nnz = 0;
            if (fmt[(uint64_t)q * S + j] == ORC_FMT_DENSE) st = orc_encode_dense(src, len, dtype, msg[q] + j * slot, slot);
            else st = orc_compress(src, len, dtype, msg[q] + j * slot, slot, &nnz);
            if (st) goto done;
        }
    }
    for (int r = 0; r < P; r++) {
        memcpy((uint8_t*)out[r] + (uint64_t)r * n * s, part[r], n * s);
        /* hop k brings rank r the stream of rank r-1-k */
        for (int k = 0; k < P - 1; k++) {
            const int q = ((r - 1 - k) % P + P) % P;
            memcpy(hop, msg[q], cap);
            st = orc_decode_sliced(hop, cap, (uint8_t*)out[r] + (uint64_t)q * n * s, n, dtype);
            if (st) goto done;
        }
    }
done:
    if (msg) for (int q = 0; q < P; q++) free(msg[q]);
    free(msg); free(hop);
    return st;
}

/* Standalone: every slice Pici (the all-gather never densifies).  fmt_out
 * (optional) gets the P * S slice formats. */
int orc_ring_all_gather_sliced(const void* const* part, void* const* out, int P, uint64_t n, int dtype,
                               uint8_t* fmt_out) {
    if (P < 1) return ORC_ERR_INVALID_ARG;
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_ERR_UNSUPPORTED;
    const uint64_t S = orc_slice_count(n);
    uint8_t* fmt = (uint8_t*)malloc((size_t)(P * S) + 1);
    if (!fmt) return ORC_ERR_INVALID_ARG;
    memset(fmt, ORC_FMT_PICI, (size_t)(P * S));
    int st = ring_all_gather_sliced_fmt(part, fmt, out, P, n, dtype);
    if (st == ORC_OK && fmt_out) memcpy(fmt_out, fmt, (size_t)(P * S));
    free(fmt);
    return st;
}

/* All-reduce: the sliced reduce-scatter, then the sliced all-gather of the
 * reduced chunks.  At the transition every slice of a rank's reduced chunk
 * extrapolates once more from that rank's slice tracker, est = sigma_prev *
 * sigma0, and goes dense iff est <= ag_thresh (Sec. IV-C per slice; adaptive
 * 0 / 2 as everywhere).  out[r] gets n elements.  fmt_rs (optional) as
 * orc_ring_reduce_scatter_sliced; fmt_ag (optional) gets the P * S slice
 * formats of the all-gather.  P = 1 sends nothing: out[0] = send[0] and the
 * formats are not written. */
int orc_ring_all_reduce_sliced(const void* const* send, void* const* out, int P, uint64_t n, int dtype,
                               const orc_policy_t* pol, uint8_t* fmt_rs, uint8_t* fmt_ag) {
    if (P < 1 || n % (uint64_t)P) return ORC_ERR_INVALID_ARG;
    if (dtype != ORC_F32 && dtype != ORC_BF16) return ORC_ERR_UNSUPPORTED;
    const uint64_t m = n / (uint64_t)P, s = elem_size(dtype), S = orc_slice_count(m);
    if (P == 1) { memcpy(out[0], send[0], n * s); return ORC_OK; }
    int st = ORC_ERR_INVALID_ARG;
    void** red = (void**)calloc((size_t)P, sizeof(void*));
    double* sig0 = (double*)calloc((size_t)(P * S + 1), sizeof(double));
    double* sigp = (double*)calloc((size_t)(P * S + 1), sizeof(double));
    uint8_t* fmt = (uint8_t*)malloc((size_t)(P * S) + 1);
    if (!red || !sig0 || !sigp || !fmt) goto done;
    for (int r = 0; r < P; r++) if (!(red[r] = malloc(m * s + 1))) goto done;
    st = rs_sliced(send, red, P, n, dtype, pol, fmt_rs, sig0, sigp);
    if (st) goto done;
    for (int r = 0; r < P; r++)
        for (uint64_t q = 0; q < S; q++) {
            const double est = sigp[r * S + q] * sig0[r * S + q];
            fmt[r * S + q] = (uint8_t)(go_dense(pol, est, pol->ag_thresh) ? ORC_FMT_DENSE : ORC_FMT_PICI);
        }
    st = ring_all_gather_sliced_fmt((const void* const*)red, fmt, out, P, m, dtype);
    if (st == ORC_OK && fmt_ag) memcpy(fmt_ag, fmt, (size_t)(P * S));
done:
    if (red) for (int r = 0; r < P; r++) free(red[r]);
    free(red); free(sig0); free(sigp); free(fmt);
    return st;
}

/* ---- timing helper of the benchmark's CPU-baseline leg ------------------ */
/* Not a definition of the method: the benchmark's step, run on the functions
 * above as they stand -- compress(a) into s1, decompress s1 into d1,
 * a (+) Pici(b) -> Pici s2, Pici(s1) (+) Pici(b) -> Pici s3,
 * a (+) Pici(b) -> dense d2, and the expansion of s1 and s2 (the all-gather
 * receive side) -- reps times on caller-owned buffers (cap bytes each for s1,
 * s2, s3; n elements each for d1, d2).  secs[r] is repetition r's time in
 * seconds (monotonic clock).  Returns the first failing status, else 0. */
static double now_s(void) {
    struct timespec ts;
    clock_gettime(CLOCK_MONOTONIC, &ts);
    return (double)ts.tv_sec + 1e-9 * (double)ts.tv_nsec;
}

int orc_time_step(const void* a, const uint8_t* b, uint64_t b_cap, uint64_t n, int dtype, uint8_t* s1,
                  uint8_t* s2, uint8_t* s3, uint64_t cap, void* d1, void* d2, int reps, double* secs) {
    for (int r = 0; r < reps; r++) {
        uint64_t nnz = 0;
        const double t0 = now_s();
        int st = orc_compress(a, n, dtype, s1, cap, &nnz);
        if (!st) st = orc_decompress(s1, cap, d1, n, dtype);
        if (!st) st = orc_reduce(ORC_ARRAY, a, n * elem_size(dtype), ORC_STREAM, b, b_cap, ORC_STREAM, ORC_FMT_PICI,
                                 s2, cap, n, dtype, &nnz);
        if (!st) st = orc_reduce(ORC_STREAM, s1, cap, ORC_STREAM, b, b_cap, ORC_STREAM, ORC_FMT_PICI, s3, cap, n,
                                 dtype, &nnz);
        if (!st) st = orc_reduce(ORC_ARRAY, a, n * elem_size(dtype), ORC_STREAM, b, b_cap, ORC_ARRAY, ORC_FMT_DENSE,
                                 d2, n * elem_size(dtype), n, dtype, &nnz);
        if (!st) st = orc_decompress(s1, cap, d1, n, dtype);
        if (!st) st = orc_decompress(s2, cap, d2, n, dtype);
        secs[r] = now_s() - t0;
        if (st) return st;
    }
    return ORC_OK;
}
