// gfx950 kernels of the Pici hot path (SpCCL, arXiv 2607.04676) and their
// host launchers.
//
// Tile mapping.  The format views the input as 64x64 row-major tiles and
// stores one 64-bit bit-vector word per tile column (Sec. III-B).  On a
// 64-lane CDNA wavefront the natural mapping is one wave per tile and one
// lane per column: lane c reads element 64r + c of row r, so each row load is
// one fully coalesced 256-byte (fp32) access, the lane assembles its column
// word on its own (no cross-lane traffic), and the per-column counts needed
// for compaction are one wave prefix scan of 64 popcounts.  (The paper's
// 32-lane warps give each thread two columns, Alg. 1; that split is not
// needed here.)
//
// One pass over the input.  Compression and the Pici-producing reductions
// read their input once: each block (four waves, four tiles = one
// partition) builds B, counts, publishes its aggregate, and either finds its
// global offset in the same launch -- from the aggregates of the partitions
// before it in its chunk of 256 and the sums of the earlier chunks, a
// two-level form of the look-back of Merrill & Garland, "Single-pass Parallel
// Prefix Scan with Decoupled Look-back", 2016 -- and writes I and A, or parks
// its values for a second (place) pass.  Values are compacted through an
// 8 KiB per-wave LDS stage and written out contiguously.
//
// Numerics.  Elements are raw bit patterns; "present" = nonzero bits.  The
// reduction adds in fp32 (bf16 operands widened exactly, the sum rounded once
// to bf16, nearest-even); an absent operand is the identity.
#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <atomic>
#include <stdint.h>


#include "spccl_internal.h"
#include "../../include/spccl.h"

namespace spccl {

// ---------------------------------------------------------------------------
// element types
// cap: values one wave can stage in LDS.  A tile with more nonzeros is
// staged in groups of group_cols columns (at most 64 values each).
constexpr uint32_t pow2_floor(uint32_t x) { return x < 2 ? x : 2 * pow2_floor(x / 2); }

struct F32 {
    using raw = uint32_t;
    static constexpr int dtype = kF32;
    static constexpr uint32_t cap = kStageBytes / 4;
    static constexpr uint32_t group_cols = pow2_floor(cap / 64);
    static constexpr int groups = 64 / group_cols;
};
struct BF16 {
    using raw = uint16_t;
    static constexpr int dtype = kBF16;
    static constexpr uint32_t cap = kStageBytes / 2;
    static constexpr uint32_t group_cols = pow2_floor(cap / 64 < 64 ? cap / 64 : 64);
    static constexpr int groups = 64 / group_cols;
};

// a (+) b on raw bits: absent (0) is the identity, otherwise add.
__device__ __forceinline__ uint32_t oplus(F32, uint32_t a, uint32_t b) {
    uint32_t s = __float_as_uint(__uint_as_float(a) + __uint_as_float(b));
    s = (a == 0u) ? b : s;
    return (b == 0u) ? a : s;
}
// bf16: the fp32 sum (exact enough: fp32 keeps at least 2 * 8 + 2 significant
// bits, so rounding it again to bf16 gives the correctly rounded bf16 sum)
// rounded to nearest even by the hardware conversion (v_cvt_pk_bf16_f32; fp32
// subnormals are kept, so bf16 subnormals round the same way).
__device__ __forceinline__ uint32_t oplus(BF16, uint32_t a, uint32_t b) {
    const float f = __uint_as_float(a << 16) + __uint_as_float(b << 16);
    uint32_t s = (uint32_t)__bfloat16_as_ushort(__float2bfloat16(f));
    s = (a == 0u) ? b : s;
    return (b == 0u) ? a : s;
}

// ---------------------------------------------------------------------------
// wave primitives
__device__ __forceinline__ uint32_t lane_id() { return __lane_id(); }

// Inclusive prefix sum over the wave's 64 lanes with DPP moves: shifts by
// 1, 2, 4, 8 inside each row of 16 lanes (lanes shifted in from outside the
// row read 0), then each row adds the total of the rows before it (row
// broadcasts of lanes 15 and 31).  No LDS traffic and no address registers.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
    constexpr int kRowShr = 0x110, kRowBcast15 = 0x142, kRowBcast31 = 0x143;
    int v = (int)x;
    v += __builtin_amdgcn_update_dpp(0, v, kRowShr + 1, 0xf, 0xf, false);
    v += __builtin_amdgcn_update_dpp(0, v, kRowShr + 2, 0xf, 0xf, false);
    v += __builtin_amdgcn_update_dpp(0, v, kRowShr + 4, 0xf, 0xf, false);
    v += __builtin_amdgcn_update_dpp(0, v, kRowShr + 8, 0xf, 0xf, false);
    v += __builtin_amdgcn_update_dpp(0, v, kRowBcast15, 0xa, 0xf, false);
    v += __builtin_amdgcn_update_dpp(0, v, kRowBcast31, 0xc, 0xf, false);
    return (uint32_t)v;
}

__device__ __forceinline__ uint32_t wave_excl_scan(uint32_t x) { return wave_incl_scan(x) - x; }

// OR of x over the wave's 64 lanes (same DPP pattern), as a scalar.
__device__ __forceinline__ uint32_t wave_or(uint32_t x) {
    constexpr int kRowShr = 0x110, kRowBcast15 = 0x142, kRowBcast31 = 0x143;
    int v = (int)x;
    v |= __builtin_amdgcn_update_dpp(0, v, kRowShr + 1, 0xf, 0xf, false);
    v |= __builtin_amdgcn_update_dpp(0, v, kRowShr + 2, 0xf, 0xf, false);
    v |= __builtin_amdgcn_update_dpp(0, v, kRowShr + 4, 0xf, 0xf, false);
    v |= __builtin_amdgcn_update_dpp(0, v, kRowShr + 8, 0xf, 0xf, false);
    v |= __builtin_amdgcn_update_dpp(0, v, kRowBcast15, 0xa, 0xf, false);
    v |= __builtin_amdgcn_update_dpp(0, v, kRowBcast31, 0xc, 0xf, false);
    return (uint32_t)__builtin_amdgcn_readlane(v, 63);
}

// x of lane `lane`, which must be the same in every lane (a scalar read).
__device__ __forceinline__ uint32_t lane_bcast(uint32_t x, uint32_t lane) {
    return (uint32_t)__builtin_amdgcn_readlane((int)x, (int)lane);
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t x) { return lane_bcast(wave_incl_scan(x), 63); }

// Order this wave's LDS accesses: a wave's LDS operations execute in order,
// so waiting for its own outstanding ones (and stopping the compiler from
// moving accesses across) is enough between lanes of one wave.
__device__ __forceinline__ void wave_lds_sync() {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_wave_barrier();
}

// Bit r set iff v[r] is nonzero.  Each half is built as a doubling chain
// from its top row down (one compare and one add-with-carry per row, written
// out so that the compiler keeps no per-row constants live).
__device__ __forceinline__ uint64_t nonzero_rows(const uint32_t (&v)[64]) {
    uint32_t hi = 0, lo = 0;
#pragma unroll
    for (int r = 63; r >= 32; r--)
        asm volatile("v_cmp_ne_u32_e32 vcc, 0, %1\n\tv_addc_co_u32_e32 %0, vcc, %0, %0, vcc"
                     : "+v"(hi) : "v"(v[r]) : "vcc");
#pragma unroll
    for (int r = 31; r >= 0; r--)
        asm volatile("v_cmp_ne_u32_e32 vcc, 0, %1\n\tv_addc_co_u32_e32 %0, vcc, %0, %0, vcc"
                     : "+v"(lo) : "v"(v[r]) : "vcc");
    return ((uint64_t)hi << 32) | lo;
}

// Streaming stores for output that is written once and read, if at all, by a
// later launch: non-temporal, so the lines go out without displacing
// anything.  A 256 MiB array is written ~20% faster this way than with
// ordinary stores (16-bit and 32-bit lanes alike).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
template <class T>
__device__ __forceinline__ void st_stream(T* p, T v) {
    __builtin_nontemporal_store(v, p);
}
__device__ __forceinline__ void st_stream(uint4* p, uint4 v) {
    const u32x4 x = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(x, reinterpret_cast<u32x4*>(p));
}

__device__ __forceinline__ void set_status(WsCtrl* ctrl, uint32_t code) {
    atomicCAS(&ctrl->status, 0u, code);
}

// ---------------------------------------------------------------------------
// message headers

struct HeaderView {
    bool ok;
    uint32_t fmt;
    uint64_t nnz;
};

// The six 64-bit words of a header (messages are 16-byte aligned).
struct HeaderWords {
    uint64_t w[6];
};

__device__ __forceinline__ HeaderWords load_header_words(const uint8_t* h) {
    const uint4* q = reinterpret_cast<const uint4*>(h);
    const uint4 x = q[0], y = q[1], z = q[2];
    return HeaderWords{{(uint64_t)x.x | ((uint64_t)x.y << 32), (uint64_t)x.z | ((uint64_t)x.w << 32),
                        (uint64_t)y.x | ((uint64_t)y.y << 32), (uint64_t)y.z | ((uint64_t)y.w << 32),
                        (uint64_t)z.x | ((uint64_t)z.y << 32), (uint64_t)z.z | ((uint64_t)z.w << 32)}};
}

// Checks a message header against the expected n / dtype (and format if
// want_fmt >= 0) and the buffer capacity; every offset must be the one the
// layout implies, so a passing header bounds every later read.
__device__ HeaderView check_header(const HeaderWords& hw, uint64_t cap, uint64_t n, int dtype, int want_fmt) {
    HeaderView v{false, 0u, 0ull};
    const uint64_t w0 = hw.w[0], hn = hw.w[1], nnz = hw.w[2], oI = hw.w[3], oA = hw.w[4], total = hw.w[5];
    const uint32_t magic = (uint32_t)w0, fmt = (uint32_t)(w0 >> 32) & 0xFFFFu, dt = (uint32_t)(w0 >> 48);
    bool ok = magic == kMagic && dt == (uint32_t)dtype && hn == n && total <= cap;
    if (want_fmt >= 0) ok = ok && fmt == (uint32_t)want_fmt;
    if (fmt == (uint32_t)kFmtPici)
        ok = ok && oI == off_I(n) && oA == off_A(n) && nnz <= n && total == oA + nnz * elem_bytes(dtype);
    else if (fmt == (uint32_t)kFmtDense)
        ok = ok && oA == kHeaderBytes && total == dense_msg_bytes(n, dtype);
    else if (fmt == (uint32_t)kFmtCoo)
        ok = ok && oI == kHeaderBytes && nnz <= n && oA == coo_off_V(nnz) && total == coo_bytes(dtype, nnz);
    else
        ok = false;
    v.ok = ok;
    v.fmt = fmt;
    v.nnz = nnz;
    return v;
}

__device__ HeaderView read_header(const uint8_t* h, uint64_t cap, uint64_t n, int dtype, int want_fmt) {
    if (cap < kHeaderBytes) return HeaderView{false, 0u, 0ull};
    return check_header(load_header_words(h), cap, n, dtype, want_fmt);
}

__device__ __forceinline__ void write_header(uint8_t* out, int fmt, int dtype, uint64_t n, uint64_t nnz,
                                             uint64_t oI, uint64_t oA, uint64_t total) {
    uint64_t* w = reinterpret_cast<uint64_t*>(out);
    w[0] = (uint64_t)kMagic | ((uint64_t)(uint32_t)fmt << 32) | ((uint64_t)(uint32_t)dtype << 48);
    w[1] = n;
    w[2] = nnz;
    w[3] = oI;
    w[4] = oA;
    w[5] = total;
}

// ---------------------------------------------------------------------------
// tile sources: fill v[r] = element (row r, column lane) of tile t

// Dense source, column `lane` of tile t, read through a buffer resource that
// covers only the tile's elements below n: the hardware range check returns 0
// for the rest, so full and partial tiles take one branch-free path.  The tile
// index is wave-uniform, so the resource sits in scalar registers and each row
// is an immediate (plus scalar) offset from one lane offset.
// first: v = x; otherwise v = v (+) x.
constexpr int kBufferWord3 = 0x00020000;   // gfx9 raw buffer: 32-bit data format, no swizzle
// Cache policy of the dense stream loads: non-temporal.  The dense operand is
// read once per launch; streaming it past the caches also spares the
// dirty lines a preceding large write left behind (a normal load would
// first have to write them back to make room).
constexpr int kStreamLoad = 2;

// Rows [R0, R1) of the tile.
template <class E, bool First, int R0 = 0, int R1 = 64>
__device__ __forceinline__ void fetch_dense(const uint8_t* base, uint64_t t, uint64_t n, uint32_t (&v)[64]) {
    using raw = typename E::raw;
    constexpr uint32_t rowb = 64 * sizeof(raw);             // bytes per tile row
    constexpr int per = 4096 / rowb;                         // rows per 4 KiB immediate range
    t = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(t >> 32)) << 32) |
        __builtin_amdgcn_readfirstlane((uint32_t)t);
    const uint64_t start = t * kTileElems;
    const uint64_t rem = start < n ? n - start : 0;
    const uint32_t bytes = (uint32_t)((rem < kTileElems ? rem : kTileElems) * sizeof(raw));
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(base) + (rem ? start : 0) * sizeof(raw), (short)0, (int)bytes, kBufferWord3);
    // an opaque lane offset: in a loop the compiler would otherwise hoist one
    // offset register per row instead of using the immediate offsets
    uint32_t lo = lane_id() * (uint32_t)sizeof(raw);
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int r = R0; r < R1; r++) {
        uint32_t x;
        if constexpr (sizeof(raw) == 4)
            x = __builtin_amdgcn_raw_buffer_load_b32(rs, lo + rowb * (r % per), 4096 * (r / per), kStreamLoad);
        else
            x = __builtin_amdgcn_raw_buffer_load_b16(rs, lo + rowb * (r % per), 4096 * (r / per), kStreamLoad);
        v[r] = First ? x : oplus(E{}, v[r], x);
    }
}

// All rows of a tile when the tile is the wave's only read (compression).
// fp32: four groups of 16 rows, each waited for before the next is issued.
// With every resident wave holding a whole 16 KiB tile in flight the device
// has over 100 MB of reads outstanding, more than it needs to stay busy, and
// reads slower; pacing took 2 us off a 256 MiB fp32 compression (62.5 ->
// 60.4 us).  A bf16 tile is half the bytes, and pacing it cost 8 us: bf16
// rows are issued at once.
template <class E>
__device__ __forceinline__ void fetch_dense_paced(const uint8_t* base, uint64_t t, uint64_t n, uint32_t (&v)[64]) {
    if constexpr (sizeof(typename E::raw) != 4) {
        fetch_dense<E, true>(base, t, n, v);
        return;
    }
    fetch_dense<E, true, 0, 16>(base, t, n, v);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    fetch_dense<E, true, 16, 32>(base, t, n, v);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    fetch_dense<E, true, 32, 48>(base, t, n, v);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    fetch_dense<E, true, 48, 64>(base, t, n, v);
}

// Pici source: B words, I offsets and A values of tile t of a checked
// message.  Values go through the wave's LDS stage (contiguous coalesced
// reads of the tile's A range), then each lane walks its column word.  A
// tile whose counts disagree with I (or overrun nnz) is treated as empty and
// flagged.  first: v = x; otherwise v = v (+) x.  The column words and
// offsets are read non-temporally, like the dense rows they travel with (a
// cached read measured 2-3 us slower per 256 MiB reduce).
struct PiciMeta {
    uint64_t w;        // this lane's column word (as loaded)
    uint32_t base;     // I[t]
    uint32_t next;     // I[t + 1]
};

template <class E>
__device__ __forceinline__ PiciMeta load_pici_meta(const uint8_t* msg, uint64_t t, uint64_t n) {
    const uint64_t* B = reinterpret_cast<const uint64_t*>(msg + kHeaderBytes);
    const uint32_t* I = reinterpret_cast<const uint32_t*>(msg + off_I(n));
    return PiciMeta{__builtin_nontemporal_load(&B[t * 64 + lane_id()]), __builtin_nontemporal_load(&I[t]),
                    __builtin_nontemporal_load(&I[t + 1])};
}

// The same through a buffer resource that ends at the message's index
// arrays (or its capacity, if smaller): any tile index reads inside the
// buffer (past the end the hardware returns zeros), so a wave without a tile
// issues the loads too and no branch makes it wait for them early.
template <class E>
__device__ __forceinline__ PiciMeta load_pici_meta_any(const uint8_t* msg, uint64_t cap, uint64_t t, uint64_t n) {
    const uint64_t end = off_A(n) < cap ? off_A(n) : cap;
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(msg), (short)0, (int)(uint32_t)end, kBufferWord3);
    t = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(t >> 32)) << 32) |
        __builtin_amdgcn_readfirstlane((uint32_t)t);
    const uint32_t ob = (uint32_t)(kHeaderBytes + 512ull * t), oi = (uint32_t)(off_I(n) + 4ull * t);
    // every offset in the per-lane part, which the range check always covers
    const auto w = __builtin_amdgcn_raw_buffer_load_b64(rs, ob + lane_id() * 8u, 0, kStreamLoad);
    const auto i2 = __builtin_amdgcn_raw_buffer_load_b64(rs, oi, 0, kStreamLoad);
    return PiciMeta{(uint64_t)w[0] | ((uint64_t)w[1] << 32), i2[0], i2[1]};
}

// Column counts and prefixes of a tile from its metadata, checked against
// I and nnz and against the array's end (a bit at a position >= n); a tile
// that fails is flagged and reads as empty.  So no value beyond n ever leaves
// a Pici source.
struct PiciCols {
    uint64_t w;
    uint32_t colpref, cnt, base;
    bool ok;           // the tile passed its checks (else it reads as empty)
};

__device__ __forceinline__ PiciCols pici_columns(PiciMeta m, uint64_t nnz, uint64_t t, uint64_t n, WsCtrl* ctrl) {
    const uint64_t T = num_tiles(n);
    uint64_t w = m.w;
    bool beyond = false;
    const uint64_t rem = n - t * kTileElems;
    if (rem < kTileElems) {                                   // last, partial tile: rows r with 64 r + l < n
        const uint32_t l = lane_id();
        const uint32_t rows = l < rem ? (uint32_t)((rem - l + 63) / 64) : 0u;
        const uint64_t valid = rows >= 64 ? ~0ull : ((1ull << rows) - 1ull);
        beyond = __any((w & ~valid) != 0ull);
    }
    uint32_t c = (uint32_t)__popcll(w);
    uint32_t colpref = wave_excl_scan(c);
    uint32_t cnt = lane_bcast(colpref + c, 63);
    const bool bad =
        beyond || (uint64_t)m.base + cnt > nnz || m.base + cnt != m.next || (t + 1 == T && (uint64_t)m.next != nnz);
    if (bad) {
        if (lane_id() == 0) set_status(ctrl, SPCCL_ERR_CORRUPT_STREAM);
        w = 0; colpref = 0; cnt = 0;
    }
    return PiciCols{w, colpref, cnt, m.base, !bad};
}

// Values staged with all loads in flight at once: up to kChunkVals values,
// kChunkSlots per lane.
constexpr uint32_t kChunkVals = 1024;
constexpr int kChunkSlots = kChunkVals / 64;

// src[0 .. cnt) into stage[0 .. cnt), kChunkVals at a time with every load
// of a chunk issued before the first is used.
template <class E>
__device__ __forceinline__ void stage_values(const typename E::raw* src, uint32_t cnt, typename E::raw* stage) {
    using raw = typename E::raw;
    const uint32_t l = lane_id();
    for (uint32_t c0 = 0; c0 < cnt; c0 += kChunkVals) {
        raw x[kChunkSlots];
#pragma unroll
        for (int j = 0; j < kChunkSlots; j++) {
            const uint32_t i = c0 + l + 64 * j;
            x[j] = i < cnt ? src[i] : (raw)0;
        }
#pragma unroll
        for (int j = 0; j < kChunkSlots; j++) {
            const uint32_t i = c0 + l + 64 * j;
            if (i < cnt) stage[i] = x[j];
        }
    }
}

// v (+)= the staged values of the columns whose words are in wm (zero for
// the other lanes), this lane's first value at stage[rank].  Rows set in no
// lane's word are skipped by a scalar test of the wave's OR of the words.
// With col (this lane's column of a full output tile), each row is also
// stored as soon as it is final, so the stores overlap the rest of the walk.
template <class E, bool First>
__device__ __forceinline__ void apply_staged(uint64_t wm, uint32_t rank, const typename E::raw* stage,
                                             uint32_t (&v)[64], typename E::raw* col = nullptr) {
    const uint32_t ulo = wave_or((uint32_t)wm), uhi = wave_or((uint32_t)(wm >> 32));
#pragma unroll
    for (int r = 0; r < 64; r++) {
        const bool bit = (wm >> r) & 1ull;
        if (((r < 32 ? ulo : uhi) >> (r & 31)) & 1u) {   // rows empty in every column cost one scalar branch
            asm volatile("");       // keeps that branch apart from the lanes' (see merge_sparse)
            if (bit) {
                const uint32_t x = stage[rank];
                rank++;
                v[r] = First ? x : oplus(E{}, v[r], x);
            }
        }
        if (col) st_stream(&col[64 * r], (typename E::raw)v[r]);
    }
}

template <class E, bool First>
__device__ __forceinline__ void expand_pici(PiciCols pc, const uint8_t* msg, uint64_t n, typename E::raw* stage,
                                            uint32_t (&v)[64]) {
    using raw = typename E::raw;
    const uint32_t l = lane_id();
    const uint64_t w = pc.w;
    const uint32_t colpref = pc.colpref, cnt = pc.cnt;
    const raw* src = reinterpret_cast<const raw*>(msg + off_A(n)) + pc.base;
    if (First) {
#pragma unroll
        for (int r = 0; r < 64; r++) v[r] = 0;
    }
    // one pass over all 64 columns when the tile's values fit the stage,
    // else one group of columns at a time
    const bool one = cnt <= E::cap;
    const int ngroups = one ? 1 : E::groups;
    const uint32_t gcols = one ? 64u : E::group_cols;
#pragma unroll 1
    for (int h = 0; h < ngroups; h++) {
        const uint32_t c0 = gcols * h, c1 = c0 + gcols;
        const uint32_t lo = one ? 0u : lane_bcast(colpref, c0);
        const uint32_t hi = (one || c1 == 64) ? cnt : lane_bcast(colpref, c1);
        stage_values<E>(src + lo, hi - lo, stage);
        wave_lds_sync();
        apply_staged<E, First>((l >= c0 && l < c1) ? w : 0ull, colpref - lo, stage, v);
        wave_lds_sync();
    }
}

// Early values of a Pici tile.  The tile's value range [I[t], I[t+1]) is
// known as soon as its offsets arrive, so when it holds at most kEarlyVals
// values they are read into registers right then, while the rest of a dense
// operand's rows are still in flight, instead of in a second round trip after
// all of them.  The range comes from the message and is not yet checked, so
// the loads go through a buffer resource that ends at the message's capacity
// (past it the hardware returns zeros); the values are used only once
// pici_columns has confirmed the range against the column words.  Like the
// column words, they are read non-temporally.
constexpr int kEarlySlots = 8;
constexpr int kEarlySplit = 32;          // dense rows issued before the early values
constexpr uint32_t kEarlyVals = 64 * kEarlySlots;
constexpr uint32_t kNotEarly = 0xFFFFFFFFu;

struct EarlyVals {
    uint32_t x[kEarlySlots];   // value l + 64 j of the range in x[j]
    uint32_t cnt;              // the range's length, or kNotEarly: not read early
};

template <class E>
__device__ __forceinline__ EarlyVals fetch_early(const uint8_t* msg, uint64_t cap, uint64_t n, const PiciMeta& m) {
    using raw = typename E::raw;
    EarlyVals e;
    const uint32_t base = __builtin_amdgcn_readfirstlane(m.base);
    const uint32_t next = __builtin_amdgcn_readfirstlane(m.next);
    e.cnt = (next >= base && next - base <= kEarlyVals) ? next - base : kNotEarly;
    const uint64_t start = off_A(n) + (uint64_t)base * sizeof(raw);
    const uint64_t avail = cap > start ? cap - start : 0ull;
    const uint64_t want = e.cnt == kNotEarly ? 0ull : (uint64_t)e.cnt * sizeof(raw);
    const uint32_t bytes = (uint32_t)(want < avail ? want : avail);
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(msg) + (bytes ? start : 0ull), (short)0, (int)bytes, kBufferWord3);
    uint32_t lo = lane_id() * (uint32_t)sizeof(raw);
    asm volatile("" : "+v"(lo));
#pragma unroll
    for (int j = 0; j < kEarlySlots; j++) {
        if constexpr (sizeof(raw) == 4)
            e.x[j] = __builtin_amdgcn_raw_buffer_load_b32(rs, lo + 64 * sizeof(raw) * j, 0, kStreamLoad);
        else
            e.x[j] = __builtin_amdgcn_raw_buffer_load_b16(rs, lo + 64 * sizeof(raw) * j, 0, kStreamLoad);
    }
    return e;
}

// v (+)= the tile from its early values when they cover it (the checked
// count equals the early range), else from the message as expand_pici does.
// With col (see apply_staged) the rows of an early tile are also stored;
// returns whether they were.
template <class E, bool First>
__device__ __forceinline__ bool expand_pici_early(PiciCols pc, const EarlyVals& e, const uint8_t* msg, uint64_t n,
                                                  typename E::raw* stage, uint32_t (&v)[64],
                                                  typename E::raw* col = nullptr) {
    using raw = typename E::raw;
    static_assert(kEarlyVals <= E::cap, "early values fit the stage");
    if (e.cnt != pc.cnt) {
        expand_pici<E, First>(pc, msg, n, stage, v);
        return false;
    }
    const uint32_t l = lane_id();
    if (First) {
#pragma unroll
        for (int r = 0; r < 64; r++) v[r] = 0;
    }
#pragma unroll
    for (int j = 0; j < kEarlySlots; j++)
        if (l + 64u * j < pc.cnt) stage[l + 64 * j] = (raw)e.x[j];
    wave_lds_sync();
    apply_staged<E, First>(pc.w, pc.colpref, stage, v, col);
    wave_lds_sync();
    return col != nullptr;
}

// The values of the rows set in w (this lane's column) in row order to
// stage[rank ...].  A row set in no lane's word costs one scalar test; the
// others are written without branching: a lane whose word lacks the row
// writes its own slot of `spare` (one per lane, so no bank conflicts).  The
// address is own + bit * (next - own), one 24-bit multiply-add, and the
// distance grows by bit: three VALU operations a row (a select would take a
// compare, a hazard wait and a move as well).
template <class E>
__device__ __forceinline__ void compact_rows(uint64_t w, uint32_t rank, const uint32_t (&v)[64],
                                             typename E::raw* stage, typename E::raw* spare) {
    using raw = typename E::raw;
    const uint32_t olo = wave_or((uint32_t)w), ohi = wave_or((uint32_t)(w >> 32));
    char* own = reinterpret_cast<char*>(spare + lane_id());
    int dist = (int)(reinterpret_cast<char*>(stage + rank) - own);    // LDS bytes: |dist| < 2^23
#pragma unroll
    for (int r = 0; r < 64; r++) {
        if (((r < 32 ? olo : ohi) >> (r & 31)) & 1u) {
            const int bit = (int)((w >> r) & 1ull);
            *reinterpret_cast<raw*>(own + __mul24(bit, dist)) = (raw)v[r];
            dist += bit * (int)sizeof(raw);
        }
    }
}

// A Pici operand's tile handed back unmerged (a dense + Pici pair read with
// its values early), for a sink that merges it itself.
struct EarlyPici {
    PiciCols pc;
    EarlyVals ev;
    const uint8_t* msg;
};

// Sparse merge of a Pici tile into a dense one for a Pici sink.  Where only
// the Pici operand is present, the sum is its value as it stands (the absent
// dense element is the identity), so such values need no arithmetic: they
// are copied from LDS straight to their output positions when the tile is
// compacted (copy_pici_only).  Only the rows where both operands are present
// are added in registers.  The work follows the nonzeros instead of the rows.
// Taken when the Pici values came early, no column holds more than
// kSparseCol of them, none is a stored zero (which reads as absent) and the
// union of both operands fits the stage below the parked Pici values;
// returns false (v untouched) otherwise.  On success w = the output's column
// word.  At six values per column the sparse merge is still the faster one;
// at 10% density (6.4 per column on average) the row-wise merge is.
constexpr uint32_t kSparseCol = 6;

struct SparseTile {
    uint64_t wa, wb;       // dense and Pici column words
    uint32_t colpref_b;    // this column's first Pici value
    uint32_t cb;           // this column's Pici values
};

template <class E>
__device__ __forceinline__ bool merge_sparse(const EarlyPici& ep, typename E::raw* stage, uint32_t (&v)[64],
                                             uint64_t& w, SparseTile& sp) {
    using raw = typename E::raw;
    static_assert(kEarlyVals < E::cap, "the Pici values park above the output");
    const PiciCols& pc = ep.pc;
    const uint32_t l = lane_id();
    const uint32_t cb = (uint32_t)__popcll(pc.w);
    if (ep.ev.cnt != pc.cnt) return false;
    bool zero = false;
#pragma unroll
    for (int j = 0; j < kEarlySlots; j++) zero = zero || (l + 64u * j < pc.cnt && ep.ev.x[j] == 0u);
    if (__any(zero) || __any(cb > kSparseCol)) return false;
    const uint64_t wa = nonzero_rows(v);
    if (wave_sum((uint32_t)__popcll(wa) + cb) > E::cap - kEarlyVals) return false;
    raw* bv = stage + (E::cap - kEarlyVals);
#pragma unroll
    for (int j = 0; j < kEarlySlots; j++)
        if (l + 64u * j < pc.cnt) bv[l + 64 * j] = (raw)ep.ev.x[j];
    wave_lds_sync();
    // rows held by both operands: add (an exact cancellation leaves the row
    // absent).  Few rows hold any: a row no lane holds twice costs one scalar
    // test (the empty asm keeps that test a scalar branch of its own; merged
    // with the lanes' test it would cost every row vector work and a branch
    // on the execution mask).
    const uint64_t ov = wa & pc.w;
    uint64_t cancelled = 0;
    const uint32_t olo = wave_or((uint32_t)ov), ohi = wave_or((uint32_t)(ov >> 32));
    if (olo | ohi) {
#pragma unroll
        for (int r = 0; r < 64; r++) {
            if (((r < 32 ? olo : ohi) >> (r & 31)) & 1u) {
                asm volatile("");
                if ((ov >> r) & 1ull) {
                    const uint32_t j = (uint32_t)__popcll(pc.w & ((1ull << r) - 1ull));
                    v[r] = oplus(E{}, v[r], (uint32_t)bv[pc.colpref + j]);
                    if (v[r] == 0u) cancelled |= 1ull << r;
                }
            }
        }
    }
    w = (wa | pc.w) & ~cancelled;
    sp = SparseTile{wa, pc.w, pc.colpref, cb};
    return true;
}

// The Pici-only values of a sparse-merged tile into their output positions
// (colpref = this column's first output value, w = the output word).
template <class E>
__device__ __forceinline__ void copy_pici_only(const SparseTile& sp, uint64_t w, uint32_t colpref,
                                               typename E::raw* stage) {
    using raw = typename E::raw;
    const raw* bv = stage + (E::cap - kEarlyVals);
    uint64_t rem = sp.wb;
    for (uint32_t j = 0; __any(j < sp.cb); j++) {
        if (j < sp.cb) {
            const uint32_t r = (uint32_t)__builtin_ctzll(rem);
            rem &= rem - 1ull;
            if (!((sp.wa >> r) & 1ull)) {
                const uint32_t dst = colpref + (uint32_t)__popcll(w & ((1ull << r) - 1ull));
                stage[dst] = bv[sp.colpref_b + j];
            }
        }
    }
}

// ---------------------------------------------------------------------------
// COO sources (Sec. II-B format: J = flat 32-bit indices, increasing; V =
// values in index order).  A tile's entries are a contiguous range of J,
// found by searching J for the tile's first element; inside the tile they
// are row-major, so row r's entries are contiguous and sorted by column.

// Lower bound of `key` in J[lo, hi) -- the first position whose index is
// >= key, hi if none -- searched by G groups of 64/G consecutive lanes, each
// group with its own key and range: every round each lane of a group probes
// one position and the group keeps the one interval between probes that
// holds the answer, so a range of length L takes about log_{64/G}(L)
// rounds of dependent loads.  J is read only inside [lo, hi).  The result
// depends only on (J, lo, hi, key), so two waves that search the same key
// over the same range agree and neighbouring tiles' ranges meet exactly
// even when J is corrupt.
template <int G>
__device__ uint32_t coo_lower_bound(const uint32_t* J, uint32_t lo, uint32_t hi, uint64_t key) {
    constexpr uint32_t W = 64 / G;
    const uint32_t l = lane_id(), j = l % W, sh = (l / W) * W;
    const uint64_t gmask = W == 64 ? ~0ull : (((1ull << W) - 1ull) << sh);
    while (__any(hi > lo)) {
        const uint32_t len = hi - lo;
        const uint32_t step = len ? (len + W - 1) / W : 1u;
        const uint32_t p = lo + j * step;
        const bool valid = len != 0 && p < hi;
        const bool ge = valid && (uint64_t)J[p] >= key;
        const uint64_t mg = __ballot(ge) & gmask, mv = __ballot(valid) & gmask;
        if (len) {
            const uint32_t nv = (uint32_t)__popcll(mv);
            const uint32_t f = mg ? (uint32_t)__builtin_ctzll(mg) - sh : nv;
            const uint32_t nlo = f == 0 ? lo : lo + (f - 1) * step + 1;
            const uint32_t nhi = f < nv ? lo + f * step : hi;
            lo = nlo;
            hi = nhi;
        }
    }
    return lo;
}

// Per-wave LDS of a COO tile expansion: row r's staged entries as a column
// mask and the stage position of the first of them.
struct CooLds {
    uint64_t rw[64];
    uint32_t rf[64];
};

constexpr uint32_t kCooChunk = 512;            // entries staged at a time (8 per lane)
constexpr int kCooSlots = kCooChunk / 64;

// popcount of the bits of w below this lane
__device__ __forceinline__ uint32_t bits_below_lane(uint64_t w) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(w >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)w, 0u));
}

// Entries [lo, lo + m) of J and V (m <= kCooChunk) into registers with
// every load in flight at once -- index x, its predecessor y (0 for the
// first) -- and the values into the stage.  With check, every index must
// lie in [first, limit) and the indices must increase strictly; returns
// false (the same in every lane) otherwise.
template <class E>
__device__ __forceinline__ bool coo_load(const uint32_t* J, const typename E::raw* V, uint32_t lo, uint32_t m,
                                         bool check, uint64_t first, uint64_t limit, typename E::raw* stage,
                                         uint32_t (&x)[kCooSlots], uint32_t (&y)[kCooSlots]) {
    using raw = typename E::raw;
    const uint32_t l = lane_id();
    raw val[kCooSlots];
#pragma unroll
    for (int q = 0; q < kCooSlots; q++) {
        const uint32_t i = l + 64 * q;
        x[q] = i < m ? J[lo + i] : 0u;
        y[q] = (i > 0 && i < m) ? J[lo + i - 1] : 0u;
        val[q] = i < m ? V[lo + i] : (raw)0;
    }
    bool bad = false;
#pragma unroll
    for (int q = 0; q < kCooSlots; q++) {
        const uint32_t i = l + 64 * q;
        if (i < m) {
            stage[i] = val[q];
            bad = bad || (check && (x[q] < first || x[q] >= limit || (i > 0 && x[q] <= y[q])));
        }
    }
    return !__any(bad);
}

// Adds the loaded entries that fall in tile t (positions i < m of the
// stage; indices checked) into v: each such lane sets bit c of row word r
// and, for the first entry of a row among the loaded ones, records the row's
// stage position; then lane c reads row r's value at rf[r] + (set bits of
// rw[r] below c).  (An all-zero v takes the entries exactly: zero is the
// identity of the reduction.)  With col (this lane's column of a full dense
// output tile, when these are the tile's last entries) each row is also
// stored as soon as it is final.
template <class E, int S>
__device__ __forceinline__ void coo_apply(const uint32_t (&x)[S], const uint32_t (&y)[S], uint32_t m, uint64_t t,
                                          const typename E::raw* stage, CooLds* cl, uint32_t (&v)[64],
                                          typename E::raw* col = nullptr) {
    const uint32_t l = lane_id();
    const uint64_t t0 = t * kTileElems;
    cl->rw[l] = 0ull;
    wave_lds_sync();
#pragma unroll
    for (int q = 0; q < S; q++) {
        const uint32_t i = l + 64 * q;
        if (i < m && x[q] >= t0 && x[q] < t0 + kTileElems) {
            const uint32_t loc = (uint32_t)(x[q] - t0), r = loc >> 6;
            atomicOr((unsigned long long*)&cl->rw[r], 1ull << (loc & 63u));
            if (i == 0 || (y[q] >> 6) != (x[q] >> 6)) cl->rf[r] = i;
        }
    }
    wave_lds_sync();
    const uint64_t myrw = cl->rw[l];
    const uint32_t myrf = cl->rf[l];
    wave_lds_sync();
    const uint64_t rows = __ballot(myrw != 0ull);          // rows holding entries: one scalar test per row
#pragma unroll
    for (int r = 0; r < 64; r++) {
        if ((rows >> r) & 1ull) {
            const uint64_t w = ((uint64_t)lane_bcast((uint32_t)(myrw >> 32), r) << 32) | lane_bcast((uint32_t)myrw, r);
            if ((w >> l) & 1ull) v[r] = oplus(E{}, v[r], (uint32_t)stage[lane_bcast(myrf, r) + bits_below_lane(w)]);
        }
        if (col) st_stream(&col[64 * r], (typename E::raw)v[r]);
    }
    wave_lds_sync();
}

// Entries [lo, hi) of J checked: every index in [first, limit), strictly
// increasing.  Uniform.
__device__ bool coo_span_ok(const uint32_t* J, uint32_t lo, uint32_t hi, uint64_t first, uint64_t limit) {
    const uint32_t l = lane_id();
    bool bad = hi < lo;
    if (!__any(bad)) {
        for (uint32_t i0 = 0; i0 < hi - lo; i0 += kCooChunk) {
            uint32_t x[kCooSlots], y[kCooSlots];
#pragma unroll
            for (int q = 0; q < kCooSlots; q++) {
                const uint32_t i = i0 + l + 64 * q;
                x[q] = i < hi - lo ? J[lo + i] : 0u;
                y[q] = (i > 0 && i < hi - lo) ? J[lo + i - 1] : 0u;
            }
#pragma unroll
            for (int q = 0; q < kCooSlots; q++) {
                const uint32_t i = i0 + l + 64 * q;
                if (i < hi - lo) bad = bad || x[q] < first || x[q] >= limit || (i > 0 && x[q] <= y[q]);
            }
        }
    }
    return !__any(bad);
}

// Entries [lo, lo + m) (m <= kCooChunk) of J and V into registers, every
// load in flight at once; with check, verified as coo_span_ok does.
template <class E>
__device__ __forceinline__ bool coo_load_pairs(const uint32_t* J, const typename E::raw* V, uint32_t lo, uint32_t m,
                                               bool check, uint64_t first, uint64_t limit,
                                               uint32_t (&x)[kCooSlots], typename E::raw (&val)[kCooSlots]) {
    const uint32_t l = lane_id();
#pragma unroll
    for (int q = 0; q < kCooSlots; q++) {
        const uint32_t i = l + 64 * q;
        x[q] = i < m ? J[lo + i] : 0u;
        val[q] = i < m ? V[lo + i] : (typename E::raw)0;
    }
    bool bad = false;
    if (check) {
#pragma unroll
        for (int q = 0; q < kCooSlots; q++) {
            // the predecessor of entry l + 64 q: lane l - 1's, or lane 63's of
            // the slot before (shuffled, not read again)
            const uint32_t up = __shfl_up(x[q], 1);
            const uint32_t wrap = q > 0 ? __shfl(x[q > 0 ? q - 1 : 0], 63) : 0u;
            const uint32_t y = l > 0 ? up : wrap;
            const uint32_t i = l + 64 * q;
            if (i < m) bad = bad || x[q] < first || x[q] >= limit || (i > 0 && x[q] <= y);
        }
    }
    return !__any(bad);
}

// Entries [lo, hi) of a checked COO message, claimed by tile t, checked:
// every index inside the tile and below n, strictly increasing.  Uniform.
__device__ bool coo_range_ok(const uint32_t* J, uint32_t lo, uint32_t hi, uint64_t t, uint64_t n) {
    const uint32_t l = lane_id();
    const uint64_t t0 = t * kTileElems, tend = t0 + kTileElems < n ? t0 + kTileElems : n;
    bool bad = hi < lo || hi - lo > kTileElems;
    if (!__any(bad)) {
        for (uint32_t i0 = 0; i0 < hi - lo; i0 += kCooChunk) {
            uint32_t x[kCooSlots], y[kCooSlots];
#pragma unroll
            for (int q = 0; q < kCooSlots; q++) {
                const uint32_t i = i0 + l + 64 * q;
                x[q] = i < hi - lo ? J[lo + i] : 0u;
                y[q] = (i > 0 && i < hi - lo) ? J[lo + i - 1] : 0u;
            }
#pragma unroll
            for (int q = 0; q < kCooSlots; q++) {
                const uint32_t i = i0 + l + 64 * q;
                if (i < hi - lo) bad = bad || x[q] < t0 || x[q] >= tend || (i > 0 && x[q] <= y[q]);
            }
        }
    }
    return !__any(bad);
}

// Tile t of a checked COO message (nnz entries) added into v.  Its entry
// range comes from the message's tile index when the call built one and both
// of the tile's index words carry the call's epoch (see k_coo_index), else it
// is searched for; a range that fits one chunk is checked as it is loaded, a
// larger one is checked in a pass of its own before any entry is used; then
// the entries are applied a chunk at a time (a row split between chunks gets
// its columns from both).  A tile that fails the checks is flagged and adds
// nothing.
template <class E>
__device__ void coo_tile(const uint8_t* msg, uint64_t nnz, const uint64_t* idx, uint32_t epoch, uint64_t t,
                         uint64_t n, typename E::raw* stage, CooLds* cl, WsCtrl* ctrl, uint32_t (&v)[64]) {
    using raw = typename E::raw;
    const uint32_t* J = reinterpret_cast<const uint32_t*>(msg + kHeaderBytes);
    const raw* V = reinterpret_cast<const raw*>(msg + coo_off_V(nnz));
    const uint64_t T = num_tiles(n);
    const uint64_t t0 = t * kTileElems, tlim = t0 + kTileElems < n ? t0 + kTileElems : n;
    uint32_t lo = 0, hi = 0;
    bool indexed = false;
    if (idx) {
        const uint64_t wl = idx[t], wh = idx[t + 1];
        const uint32_t el = __builtin_amdgcn_readfirstlane((uint32_t)(wl >> 32));
        const uint32_t eh = __builtin_amdgcn_readfirstlane((uint32_t)(wh >> 32));
        indexed = el == epoch && eh == epoch;
        lo = __builtin_amdgcn_readfirstlane((uint32_t)wl);
        hi = __builtin_amdgcn_readfirstlane((uint32_t)wh);
    }
    if (!indexed) {
        const uint64_t key = (lane_id() < 32 ? t : t + 1) * kTileElems;
        const uint32_t b = coo_lower_bound<2>(J, 0u, (uint32_t)nnz, key);
        lo = lane_bcast(b, 0);
        hi = lane_bcast(b, 32);
    }
    bool ok = hi >= lo && hi - lo <= kTileElems && hi <= nnz && (t > 0 || lo == 0) && (t + 1 < T || hi == nnz);
    const bool one = ok && hi - lo <= kCooChunk;
    if (ok && !one) ok = coo_range_ok(J, lo, hi, t, n);
    const uint32_t cnt = ok ? hi - lo : 0u;
    uint32_t x[kCooSlots], y[kCooSlots];
#pragma unroll 1
    for (uint32_t i0 = 0; i0 < cnt; i0 += kCooChunk) {
        const uint32_t m = cnt - i0 < kCooChunk ? cnt - i0 : kCooChunk;
        if (!coo_load<E>(J, V, lo + i0, m, one, t0, tlim, stage, x, y)) {
            ok = false;                    // only a single-chunk range is checked here: nothing applied yet
            break;
        }
        coo_apply<E>(x, y, m, t, stage, cl, v);
    }
    if (!ok && lane_id() == 0) set_status(ctrl, SPCCL_ERR_CORRUPT_STREAM);
}

// Early entries of a COO tile combined with dense rows.  The tile's entry
// range comes from the call's tile index, which lives in the workspace and
// needs no header, so when the range holds at most kCooEarly entries they are
// read into registers while the dense rows are in flight.  The header that
// places V is checked only afterwards, so these reads go through buffer
// resources that end at the message's capacity (and the index's through one
// that is empty without an index); the entries are used only once the header
// and both index words have checked out.
constexpr int kCooEarlySlots = 2;
constexpr uint32_t kCooEarly = 64 * kCooEarlySlots;

struct CooEarly {
    uint32_t x[kCooEarlySlots];     // index l + 64 q of the range
    uint32_t val[kCooEarlySlots];   // its value's bits
    uint32_t lo, hi;                // the range, from the index
    bool ok;                        // both index words carry the call's epoch and the range fits
};

// The tile's index words (issue first: the range is needed mid-way).
__device__ __forceinline__ void coo_index_words(const DevOperand& c, uint64_t t, uint64_t T, uint32_t (&w)[4]) {
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint64_t*>(c.idx), (short)0, c.idx ? (int)(8 * (T + 1)) : 0, kBufferWord3);
    const uint32_t o = (uint32_t)(8 * t);
#pragma unroll
    for (int k = 0; k < 4; k++) w[k] = __builtin_amdgcn_raw_buffer_load_b32(rs, o + 4 * k, 0, 0);
}

template <class E>
__device__ __forceinline__ CooEarly fetch_coo_early(const DevOperand& c, const HeaderWords& hw,
                                                    const uint32_t (&w)[4]) {
    using raw = typename E::raw;
    CooEarly e;
    const uint32_t lo = __builtin_amdgcn_readfirstlane(w[0]), el = __builtin_amdgcn_readfirstlane(w[1]);
    const uint32_t hi = __builtin_amdgcn_readfirstlane(w[2]), eh = __builtin_amdgcn_readfirstlane(w[3]);
    e.lo = lo;
    e.hi = hi;
    e.ok = c.idx != nullptr && el == c.idx_epoch && eh == c.idx_epoch && hi >= lo && hi - lo <= kCooEarly;
    const uint64_t m = e.ok ? hi - lo : 0u;
    const uint64_t js = kHeaderBytes + 4ull * lo, vs = hw.w[4] + (uint64_t)lo * sizeof(raw);
    const uint64_t ja = c.cap > js ? c.cap - js : 0ull, va = c.cap > vs ? c.cap - vs : 0ull;
    const uint32_t jb = (uint32_t)(4 * m < ja ? 4 * m : ja), vb = (uint32_t)(m * sizeof(raw) < va ? m * sizeof(raw) : va);
    const __amdgpu_buffer_rsrc_t rj = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(c.data) + (jb ? js : 0ull), (short)0, (int)jb, kBufferWord3);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(c.data) + (vb ? vs : 0ull), (short)0, (int)vb, kBufferWord3);
    uint32_t lj = lane_id() * 4u, lv = lane_id() * (uint32_t)sizeof(raw);
    asm volatile("" : "+v"(lj), "+v"(lv));
#pragma unroll
    for (int q = 0; q < kCooEarlySlots; q++) {
        e.x[q] = __builtin_amdgcn_raw_buffer_load_b32(rj, lj + 256 * q, 0, kStreamLoad);
        if constexpr (sizeof(raw) == 4)
            e.val[q] = __builtin_amdgcn_raw_buffer_load_b32(rv, lv + 64 * sizeof(raw) * q, 0, kStreamLoad);
        else
            e.val[q] = __builtin_amdgcn_raw_buffer_load_b16(rv, lv + 64 * sizeof(raw) * q, 0, kStreamLoad);
    }
    return e;
}

// v (+)= tile t of a checked COO message from its early entries when they
// cover the tile, else as coo_tile does.  The early range gets coo_tile's
// checks: its place in the message, and every entry inside the tile and
// above its predecessor.  With col (see coo_apply) the rows of an early tile
// are also stored; returns whether they were.
template <class E>
__device__ bool coo_tile_early(const DevOperand& c, uint64_t nnz, const CooEarly& e, uint64_t t, uint64_t n,
                               typename E::raw* stage, CooLds* cl, WsCtrl* ctrl, uint32_t (&v)[64],
                               typename E::raw* col = nullptr) {
    if (!e.ok) {
        coo_tile<E>(c.data, nnz, c.idx, c.idx_epoch, t, n, stage, cl, ctrl, v);
        return false;
    }
    const uint32_t l = lane_id();
    const uint64_t T = num_tiles(n);
    const uint64_t t0 = t * kTileElems, tlim = t0 + kTileElems < n ? t0 + kTileElems : n;
    const uint32_t lo = e.lo, hi = e.hi, m = hi - lo;
    const bool ok = hi <= nnz && (t > 0 || lo == 0) && (t + 1 < T || hi == nnz);
    uint32_t y[kCooEarlySlots];
    bool bad = false;
#pragma unroll
    for (int q = 0; q < kCooEarlySlots; q++) {
        // the predecessor of entry l + 64 q: lane l - 1's, or lane 63's of the slot before
        const uint32_t up = __shfl_up(e.x[q], 1);
        const uint32_t wrap = q > 0 ? __shfl(e.x[q > 0 ? q - 1 : 0], 63) : 0u;
        y[q] = l > 0 ? up : wrap;
        const uint32_t i = l + 64 * q;
        if (i < m) {
            stage[i] = (typename E::raw)e.val[q];
            bad = bad || e.x[q] < t0 || e.x[q] >= tlim || (i > 0 && e.x[q] <= y[q]);
        }
    }
    if (!ok || __any(bad)) {
        if (l == 0) set_status(ctrl, SPCCL_ERR_CORRUPT_STREAM);
        return false;
    }
    coo_apply<E>(e.x, y, m, t, stage, cl, v, col);
    return col != nullptr;
}

// Tile t of a (+) b into v[64] (sources: dense rows or Pici tiles; b may be
// absent).  Every read that needs no header -- the headers themselves, dense
// rows, Pici column words and offsets -- is issued first; the headers are
// checked while those are in flight, and only then are Pici values read,
// since their offsets come from the message.  The host guarantees that a
// STREAM operand's capacity covers a dense message's values or a Pici
// message's index arrays, so the early reads stay inside the caller's
// buffers whatever the header says.  Returns false, the same in every wave
// of the grid, when a header fails its check (and flags it once).
// A dense sink passes col (this lane's column of the output tile when the
// tile is full): a Pici operand read early then stores the rows as they are
// finished, and *stored says so.
// HandBack (a dense + Pici pair only): the Pici tile is not merged but
// returned, for the caller to merge.
struct PairLoad {
    bool ok;              // both headers passed (uniform over the grid)
    EarlyPici ep;         // HandBack: the unmerged Pici tile
};

template <class E, int SA, int SB, bool HandBack>
__device__ __forceinline__ PairLoad load_tile_pair_core(const DevOperand& a, const DevOperand& b, uint64_t t,
                                                        bool has_tile, uint64_t n, typename E::raw* stage,
                                                        CooLds* cl, WsCtrl* ctrl, uint32_t (&v)[64],
                                                        typename E::raw* col, bool* stored) {
    PairLoad res{true, EarlyPici{}};
    const bool ha = a.hdr != nullptr;
    const bool hb = SB != SRC_NONE && b.hdr != nullptr;
    HeaderWords hwa{}, hwb{};
    if (ha) hwa = load_header_words(a.hdr);
    if (hb) hwb = load_header_words(b.hdr);
    PiciMeta ma{0, 0, 0}, mb{0, 0, 0};
    // one dense and one Pici operand: the Pici tile's values are read early,
    // between the two halves of the dense rows
    constexpr bool early_a = SA == SRC_PICI && SB == SRC_DENSE;
    constexpr bool early_b = SA == SRC_DENSE && SB == SRC_PICI;
    // one dense and one COO operand: the COO tile's entries likewise
    constexpr bool coo_early_a = SA == SRC_COO && SB == SRC_DENSE;
    constexpr bool coo_early_b = SA == SRC_DENSE && SB == SRC_COO;
    EarlyVals ev{{0u}, kNotEarly};
    CooEarly ce{};
    if (has_tile) {
        if constexpr (SA == SRC_PICI) ma = load_pici_meta<E>(a.data, t, n);
        if constexpr (SB == SRC_PICI) mb = load_pici_meta<E>(b.data, t, n);
        asm volatile("" ::: "memory");
        if constexpr (early_a || early_b) {
            const uint8_t* d = early_b ? a.data : b.data;
            fetch_dense<E, true, 0, kEarlySplit>(d, t, n, v);
            asm volatile("" ::: "memory");
            ev = early_b ? fetch_early<E>(b.data, b.cap, n, mb) : fetch_early<E>(a.data, a.cap, n, ma);
            asm volatile("" ::: "memory");
            fetch_dense<E, true, kEarlySplit, 64>(d, t, n, v);
        } else if constexpr (coo_early_a || coo_early_b) {
            const DevOperand& c = coo_early_b ? b : a;
            uint32_t iw[4];
            coo_index_words(c, t, num_tiles(n), iw);
            asm volatile("" ::: "memory");
            fetch_dense<E, true, 0, kEarlySplit>(coo_early_b ? a.data : b.data, t, n, v);
            asm volatile("" ::: "memory");
            ce = fetch_coo_early<E>(c, coo_early_b ? hwb : hwa, iw);
            asm volatile("" ::: "memory");
            fetch_dense<E, true, kEarlySplit, 64>(coo_early_b ? a.data : b.data, t, n, v);
        } else {
            if constexpr (SA == SRC_DENSE && SB == SRC_NONE) {
                fetch_dense_paced<E>(a.data, t, n, v);
            } else {
                if constexpr (SA == SRC_DENSE) fetch_dense<E, true>(a.data, t, n, v);
                if constexpr (SB == SRC_DENSE) fetch_dense<E, SA != SRC_DENSE>(b.data, t, n, v);
            }
        }
    }
    bool ok = true;
    uint64_t nnza = 0, nnzb = 0;
    constexpr int fa = SA == SRC_PICI ? kFmtPici : (SA == SRC_COO ? kFmtCoo : kFmtDense);
    constexpr int fb = SB == SRC_PICI ? kFmtPici : (SB == SRC_COO ? kFmtCoo : kFmtDense);
    if (ha) {
        const HeaderView h = check_header(hwa, a.cap, n, E::dtype, fa);
        ok = ok && h.ok;
        nnza = h.nnz;
    }
    if (hb) {
        const HeaderView h = check_header(hwb, b.cap, n, E::dtype, fb);
        ok = ok && h.ok;
        nnzb = h.nnz;
    }
    if (!ok) {
        if (blockIdx.x == 0 && threadIdx.x == 0) set_status(ctrl, SPCCL_ERR_CORRUPT_STREAM);
        res.ok = false;
        return res;
    }
    if (has_tile) {
        constexpr bool dense_first = SA == SRC_DENSE || SB == SRC_DENSE;
        constexpr bool a_sparse = SA == SRC_PICI || SA == SRC_COO;
        if constexpr (early_a) {
            const PiciCols pc = pici_columns(ma, nnza, t, n, ctrl);
            if constexpr (HandBack) {
                res.ep = EarlyPici{pc, ev, a.data};
            } else {
                const bool st = expand_pici_early<E, false>(pc, ev, a.data, n, stage, v, col);
                if (stored) *stored = st;
            }
        }
        else if constexpr (SA == SRC_PICI)
            expand_pici<E, !dense_first>(pici_columns(ma, nnza, t, n, ctrl), a.data, n, stage, v);
        if constexpr (SA == SRC_COO) {
            if (!dense_first) {
#pragma unroll
                for (int r = 0; r < 64; r++) v[r] = 0;
            }
            if constexpr (coo_early_a) {
                const bool st = coo_tile_early<E>(a, nnza, ce, t, n, stage, cl, ctrl, v, col);
                if (stored) *stored = st;
            } else
                coo_tile<E>(a.data, nnza, a.idx, a.idx_epoch, t, n, stage, cl, ctrl, v);
        }
        if constexpr (early_b) {
            const PiciCols pc = pici_columns(mb, nnzb, t, n, ctrl);
            if constexpr (HandBack) {
                res.ep = EarlyPici{pc, ev, b.data};
            } else {
                const bool st = expand_pici_early<E, false>(pc, ev, b.data, n, stage, v, col);
                if (stored) *stored = st;
            }
        }
        else if constexpr (SB == SRC_PICI)
            expand_pici<E, !dense_first && !a_sparse>(pici_columns(mb, nnzb, t, n, ctrl), b.data, n, stage, v);
        if constexpr (SB == SRC_COO) {
            if (!dense_first && !a_sparse) {
#pragma unroll
                for (int r = 0; r < 64; r++) v[r] = 0;
            }
            if constexpr (coo_early_b) {
                const bool st = coo_tile_early<E>(b, nnzb, ce, t, n, stage, cl, ctrl, v, col);
                if (stored) *stored = st;
            } else
                coo_tile<E>(b.data, nnzb, b.idx, b.idx_epoch, t, n, stage, cl, ctrl, v);
        }
    }
    return res;
}

template <class E, int SA, int SB>
__device__ __forceinline__ bool load_tile_pair(const DevOperand& a, const DevOperand& b, uint64_t t, bool has_tile,
                                               uint64_t n, typename E::raw* stage, CooLds* cl, WsCtrl* ctrl,
                                               uint32_t (&v)[64], typename E::raw* col = nullptr,
                                               bool* stored = nullptr) {
    return load_tile_pair_core<E, SA, SB, false>(a, b, t, has_tile, n, stage, cl, ctrl, v, col, stored).ok;
}

// ---------------------------------------------------------------------------
// look-back words and the two-level offset search

constexpr uint32_t kFlagAggregate = 1, kFlagPrefix = 2;
constexpr uint32_t kSpinLimit = 1u << 20;

__device__ __forceinline__ void publish(uint64_t* flags, uint32_t p, uint32_t epoch30, uint32_t state, uint32_t val) {
    const uint64_t f = ((uint64_t)epoch30 << 34) | ((uint64_t)state << 32) | (uint64_t)val;
    __hip_atomic_store(&flags[p], f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// No exclusive prefix: a wait ran out (an offset is below 2^32 - 1, since
// n < 2^32).
constexpr uint32_t kNoPrefix = 0xFFFFFFFFu;

// Exclusive prefix of partition p in two levels, computed by one whole wave
// once p has published its own aggregate `agg` (flags[p]): the aggregates of
// the partitions before p in its chunk of kPlaceChunk (four per lane) and the
// sums of the earlier chunks (flags[nparts + c]; the first 64 loaded in the
// same round trip, one per lane), each reloaded until it carries this call's
// epoch.  A chunk's last partition publishes its chunk's sum as soon as it has
// the chunk's aggregates, before it waits for anything else.  A wave waits
// only for lower-numbered partitions, which publish their aggregates before
// they wait, and work-groups start in index order, so every wait ends; the
// spin limit bounds it regardless (ok = false, TIMEOUT set).
__device__ uint32_t chunk_lookback(uint64_t* flags, uint32_t nparts, uint32_t p, uint32_t agg, uint32_t epoch30,
                                   WsCtrl* ctrl, bool& ok) {
    constexpr int J = (int)(kPlaceChunk / 64);
    const uint32_t l = lane_id();
    const uint32_t chunk = p / kPlaceChunk, first = chunk * kPlaceChunk;
    const bool last_of_chunk = p % kPlaceChunk == kPlaceChunk - 1 || p == nparts - 1;
    ok = true;
    uint64_t fq[J];
    bool ready[J];
#pragma unroll
    for (int j = 0; j < J; j++) {
        ready[j] = first + l + 64u * j >= p;
        fq[j] = 0;
    }
    uint64_t fk = 0;
    bool kready = l >= chunk;                        // lane l: the sum of chunk l
    bool local_done = false;
    uint32_t local = 0, spins = 0;
    while (true) {
        bool all = true;
#pragma unroll
        for (int j = 0; j < J; j++) {
            if (!ready[j]) {
                fq[j] = __hip_atomic_load(&flags[first + l + 64u * j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                ready[j] = (uint32_t)(fq[j] >> 34) == epoch30;
            }
            all = all && ready[j];
        }
        if (!kready) {
            fk = __hip_atomic_load(&flags[nparts + l], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            kready = (uint32_t)(fk >> 34) == epoch30;
        }
        if (!local_done && __all(all)) {
            local_done = true;
#pragma unroll
            for (int j = 0; j < J; j++) local += first + l + 64u * j < p ? (uint32_t)fq[j] : 0u;
            local = wave_sum(local);
            if (last_of_chunk && l == 0) publish(flags, nparts + chunk, epoch30, kFlagAggregate, local + agg);
        }
        if (local_done && __all(kready)) break;
        if (++spins > kSpinLimit) {
            ok = false;
            break;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    uint32_t base = l < chunk ? (uint32_t)fk : 0u;
    // chunks 64 and beyond (outputs of more than 16384 partitions), 64 per round
    for (uint32_t k0 = 64; k0 < chunk && ok; k0 += 64) {
        const uint32_t k = k0 + l;
        uint64_t fk2 = 0;
        bool ready2 = k >= chunk;
        uint32_t spins2 = 0;
        while (true) {
            if (!ready2) {
                fk2 = __hip_atomic_load(&flags[nparts + k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                ready2 = (uint32_t)(fk2 >> 34) == epoch30;
            }
            if (__all(ready2)) break;
            if (++spins2 > kSpinLimit) {
                ok = false;
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        base += k < chunk ? (uint32_t)fk2 : 0u;
    }
    if (!ok && l == 0) set_status(ctrl, SPCCL_ERR_TIMEOUT);
    return wave_sum(base) + local;
}

// ---------------------------------------------------------------------------
// Pici sink: out = Pici(srcA (+) srcB).

// Deferred = false: one launch; each partition finds its global offset with
// chunk_lookback and writes its values in place.
// Deferred = true: first of two passes; each partition publishes its
// aggregate, writes B and the tile offsets relative to the partition, and
// parks its compacted values in its own worst-case slot of the workspace,
// never waiting on another block; k_place then moves each slot into place.
template <class E, int SA, int SB, bool Deferred>
__device__ __forceinline__ void to_pici_body(const PiciSinkArgs& g) {
    using raw = typename E::raw;
    __shared__ raw stage_all[kWavesPerBlock][E::cap];
    __shared__ raw spare_all[kWavesPerBlock][64];         // compact_rows' per-lane slots
    __shared__ uint32_t s_cnt[kWavesPerBlock];
    __shared__ uint32_t s_prefix;

    const uint32_t wave = threadIdx.x >> 6, l = lane_id();
    raw* stage = stage_all[wave];
    // Partition = block index.  Work-groups start in index order on each XCD,
    // so the lowest unfinished partition is always resident and every wait
    // below ends (the spin limit bounds it regardless).
    const uint32_t p = blockIdx.x;
    const uint32_t epoch30 = g.epoch & 0x3FFFFFFFu;
    const uint64_t t = (uint64_t)p * kTilesPerPart + wave;
    const bool has_tile = t < g.T;

    // a dense and a Pici operand: the Pici tile comes back unmerged and is
    // merged sparsely when it can be (merge_sparse)
    constexpr bool dense_pici = (SA == SRC_DENSE && SB == SRC_PICI) || (SA == SRC_PICI && SB == SRC_DENSE);
    uint32_t v[64];
    const PairLoad pl =
        load_tile_pair_core<E, SA, SB, dense_pici>(g.a, g.b, t, has_tile, g.n, stage, nullptr, g.ctrl, v, nullptr,
                                                   nullptr);
    if (!pl.ok) return;           // uniform over the grid: no partition publishes
    const EarlyPici& ep = pl.ep;
    uint64_t w = 0;
    uint32_t c = 0;
    bool sparse = false;
    SparseTile sp{};
    if (has_tile) {
        // every source reads as zero at positions >= n (bounded buffer loads,
        // Pici tiles checked against the array's end)
        if constexpr (dense_pici) {
            sparse = merge_sparse<E>(ep, stage, v, w, sp);
            if (!sparse) {
                expand_pici_early<E, false>(ep.pc, ep.ev, ep.msg, g.n, stage, v);
                w = nonzero_rows(v);
            }
        } else {
            w = nonzero_rows(v);
        }
        c = (uint32_t)__popcll(w);
        st_stream(&reinterpret_cast<uint64_t*>(g.out + kHeaderBytes)[t * 64 + l], w);
    }
    const uint32_t colpref = wave_excl_scan(c);
    const uint32_t tilecnt = lane_bcast(colpref + c, 63);
    if (l == 0) s_cnt[wave] = tilecnt;
    __syncthreads();

    uint32_t tile_excl = 0, agg = 0;
#pragma unroll
    for (uint32_t k = 0; k < kWavesPerBlock; k++) {
        const uint32_t ck = s_cnt[k];
        tile_excl += k < wave ? ck : 0u;
        agg += ck;
    }
    if (threadIdx.x == 0) publish(g.flags, p, epoch30, kFlagAggregate, agg);

    const bool single = tilecnt <= E::cap;        // always so for a sparse-merged tile
    if (has_tile && single) {
        // every output row in order (a sparse-merged tile writes zeros into
        // its Pici-only rows here, then their values over them)
        compact_rows<E>(w, colpref, v, stage, spare_all[wave]);
        if (sparse) copy_pici_only<E>(sp, w, colpref, stage);
    }
    if constexpr (Deferred) {
        if (!has_tile) return;
        // parked values are re-read by the place pass right after: ordinary
        // stores keep them in the caches (streaming ones cost 14 us at sigma 0.9)
        raw* slot = reinterpret_cast<raw*>(g.slots) + (uint64_t)p * kPartElems + tile_excl;
        if (single) {
            wave_lds_sync();
            for (uint32_t i = l; i < tilecnt; i += 64) slot[i] = stage[i];
        } else {
#pragma unroll
            for (int h = 0; h < E::groups; h++) {
                const uint32_t lo = lane_bcast(colpref, E::group_cols * h);
                const uint32_t hi = h == E::groups - 1 ? tilecnt : lane_bcast(colpref, E::group_cols * (h + 1));
                const bool mine = l / E::group_cols == (uint32_t)h;
                uint32_t rank = colpref - lo;
#pragma unroll
                for (int r = 0; r < 64; r++)
                    if (__any(mine && v[r] != 0u)) {
                        if (mine && v[r] != 0u) { stage[rank] = (raw)v[r]; rank++; }
                    }
                wave_lds_sync();
                for (uint32_t i = l; i < hi - lo; i += 64) slot[lo + i] = stage[i];
                wave_lds_sync();
            }
        }
        if (l == 0) reinterpret_cast<uint32_t*>(g.out + off_I(g.n))[t] = tile_excl;   // k_place adds the prefix
        return;
    }
    if (wave == 0) {
        bool ok;
        const uint32_t prefix = chunk_lookback(g.flags, g.nparts, p, agg, epoch30, g.ctrl, ok);
        if (l == 0) s_prefix = ok ? prefix : kNoPrefix;
    }
    __syncthreads();

    const uint32_t prefix = s_prefix;
    if (prefix == kNoPrefix) return;            // a predecessor never published: write nothing
    const uint64_t oI = off_I(g.n), oA = off_A(g.n);
    raw* A = reinterpret_cast<raw*>(g.out + oA);
    const uint32_t tbase = prefix + tile_excl;
    if (has_tile) {
        if (single) {
            raw* dst = A + tbase;
            for (uint32_t i = l; i < tilecnt; i += 64) st_stream(&dst[i], stage[i]);
        } else {
#pragma unroll
            for (int h = 0; h < E::groups; h++) {
                const uint32_t lo = lane_bcast(colpref, E::group_cols * h);
                const uint32_t hi = h == E::groups - 1 ? tilecnt : lane_bcast(colpref, E::group_cols * (h + 1));
                const bool mine = l / E::group_cols == (uint32_t)h;
                uint32_t rank = colpref - lo;
#pragma unroll
                for (int r = 0; r < 64; r++)
                    if (__any(mine && v[r] != 0u)) {
                        if (mine && v[r] != 0u) { stage[rank] = (raw)v[r]; rank++; }
                    }
                wave_lds_sync();
                raw* dst = A + tbase + lo;
                for (uint32_t i = l; i < hi - lo; i += 64) st_stream(&dst[i], stage[i]);
                wave_lds_sync();
            }
        }
        if (l == 0) reinterpret_cast<uint32_t*>(g.out + oI)[t] = tbase;
    }
    if (p == g.nparts - 1 && threadIdx.x == 0) {
        const uint64_t nnz = (uint64_t)prefix + agg;
        uint32_t* I = reinterpret_cast<uint32_t*>(g.out + oI);
        I[g.T] = (uint32_t)nnz;
        for (uint64_t b = oI + 4 * (g.T + 1); b < oA; b += 4) *reinterpret_cast<uint32_t*>(g.out + b) = 0u;
        write_header(g.out, kFmtPici, E::dtype, g.n, nnz, oI, oA, oA + nnz * sizeof(raw));
    }
}

// The count pass of a compression holds five waves per SIMD (96 VGPRs, no
// spills; the stage size keeps five blocks within the LDS): 3-6 us faster on a
// 256 MiB bf16 compression at sigma 0.9.  The reducing sinks keep four: at
// five they spill.
constexpr int sink_waves(int sb, bool deferred) { return (sb == SRC_NONE && deferred) ? 5 : 1; }

template <class E, int SA, int SB, bool Deferred>
__global__ void __launch_bounds__(kBlockThreads, sink_waves(SB, Deferred)) k_to_pici(PiciSinkArgs g) {
    to_pici_body<E, SA, SB, Deferred>(g);
}

// One ring step's Pici outputs for a batch of ranks (grid y), in one launch
// or as the count pass.  Work-groups start in order of the flattened block
// index, so a rank's blocks start after those of lower ranks, and a block
// waits only for lower partitions of its own rank.
template <class E, int SA, int SB, bool Deferred>
__global__ void __launch_bounds__(kBlockThreads, sink_waves(SB, Deferred)) k_to_pici_rb(PiciSinkArgs g, RankBatch rb) {
    if (rank_skipped(rb, blockIdx.y)) return;
    to_pici_body<E, SA, SB, Deferred>(rank_sink(g, rb, blockIdx.y));
}


// ---------------------------------------------------------------------------
// Pici (+) Pici -> Pici with work proportional to the nonzeros.
//
// Phase 1 finds each output column word: the operands' values for a group of
// columns are staged in LDS (a's run, then b's run), and rows held by both
// operands are added to find exact cancellations (every row of the group is
// checked if a staged value is itself zero, which reads as absent).  Once the
// tile's destination is known (its slot in the two-pass mode, the look-back
// prefix in the single-pass mode), phase 2 merges each column's two runs in
// row order and each lane stores its column's results in place.  A tile
// whose two value ranges fit kChunkVals together is one group of 64 columns,
// read with all loads in flight at once and staged a single time; denser
// tiles go through in groups of PPGroup::cols columns, staged again in
// phase 2.
struct PPGroup {
    static constexpr uint32_t cols = kChunkVals / 128;        // 2 operands x 64 rows per column
    static constexpr int count = 64 / cols;
};

// Whether staging round j (lanes' j-th values) holds any of `count` values.
// 32-bit values skip empty rounds behind a uniform branch; 16-bit ones take
// every round, since behind such branches their loads were each waited for
// before the next was issued (measured: bf16 Pici (+) Pici at sigma 0.9,
// 2^27 elements, 119 -> 155 us).
template <class E>
__device__ __forceinline__ bool stage_round(int j, uint32_t count) {
    return sizeof(typename E::raw) != 4 || 64u * (uint32_t)j < count;
}

// The value ranges of columns [c0, c1) of both operands into in[]: a's at
// [0, la), b's at [la, la + lb) (la + lb <= kChunkVals), every load issued
// before the first is used.  Returns la; zero = some staged value has
// all-zero bits (uniform over the wave).
template <class E>
__device__ __forceinline__ uint32_t pp_stage(const PiciCols& ca, const PiciCols& cb, const typename E::raw* pa,
                                             const typename E::raw* pb, uint32_t c0, uint32_t c1,
                                             typename E::raw* in, bool& zero) {
    using raw = typename E::raw;
    const uint32_t l = lane_id();
    const uint32_t a0 = lane_bcast(ca.colpref, c0);
    const uint32_t a1 = c1 == 64 ? ca.cnt : lane_bcast(ca.colpref, c1);
    const uint32_t b0 = lane_bcast(cb.colpref, c0);
    const uint32_t b1 = c1 == 64 ? cb.cnt : lane_bcast(cb.colpref, c1);
    const uint32_t la = a1 - a0, lb = b1 - b0;
    raw x[kChunkSlots];
#pragma unroll
    for (int j = 0; j < kChunkSlots; j++) {
        const uint32_t i = l + 64 * j;
        x[j] = (raw)1;
        if (stage_round<E>(j, la + lb)) x[j] = i < la ? pa[a0 + i] : (i < la + lb ? pb[b0 + (i - la)] : (raw)1);
    }
    bool z = false;
#pragma unroll
    for (int j = 0; j < kChunkSlots; j++) {
        const uint32_t i = l + 64 * j;
        if (stage_round<E>(j, la + lb)) {
            z |= x[j] == 0;
            if (i < la + lb) in[i] = x[j];
        }
    }
    zero = __any(z);
    wave_lds_sync();
    return la;
}

// Cancellations (exact zero sums) among the rows of this lane's column held by
// both operands -- or by either one when `zero` says a staged value is itself
// zero -- with a's run at in[ra ...] and b's at in[rb ...].  Branch-free over
// the lane's rows: each round takes the lowest row still to check (no row for
// a lane that is done: it reads in[0] and changes nothing).
template <class E>
__device__ __forceinline__ uint64_t pp_cancel(uint64_t wa, uint64_t wb, const typename E::raw* in, uint32_t ra,
                                              uint32_t rb, bool zero, bool mine) {
    uint64_t chk = mine ? (zero ? (wa | wb) : (wa & wb)) : 0ull;
    uint64_t cancel = 0;
    while (__any(chk != 0ull)) {
        const uint64_t bit = chk & (0ull - chk);
        chk ^= bit;
        const uint64_t below = bit - 1ull;
        const bool ha = (wa & bit) != 0ull, hb = (wb & bit) != 0ull;
        const uint32_t va = (uint32_t)in[ha ? ra + (uint32_t)__popcll(wa & below) : 0u];
        const uint32_t vb = (uint32_t)in[hb ? rb + (uint32_t)__popcll(wb & below) : 0u];
        const uint32_t x = oplus(E{}, ha ? va : 0u, hb ? vb : 0u);
        cancel |= x == 0u ? bit : 0ull;
    }
    return cancel;
}

// Row-order merge of this lane's two runs (a's at in[ia ...], b's at
// in[ib ...]); results present in wo go to dst[k ...].  Each round takes the
// lane's lowest remaining row: the two reads and the run positions advance
// without branches (a lane that is done reads in[0] and changes nothing),
// only the store is predicated.
template <class E>
__device__ __forceinline__ void pp_merge(uint64_t wa, uint64_t wb, uint64_t wo, const typename E::raw* in,
                                         uint32_t ia, uint32_t ib, typename E::raw* dst, uint32_t k, bool mine) {
    uint64_t todo = mine ? (wa | wb) : 0ull;
    while (__any(todo != 0ull)) {
        const uint64_t bit = todo & (0ull - todo);
        todo ^= bit;
        const bool ha = (wa & bit) != 0ull, hb = (wb & bit) != 0ull;
        const uint32_t va = (uint32_t)in[ha ? ia : 0u];
        const uint32_t vb = (uint32_t)in[hb ? ib : 0u];
        ia += ha ? 1u : 0u;
        ib += hb ? 1u : 0u;
        const uint32_t x = oplus(E{}, ha ? va : 0u, hb ? vb : 0u);
        if ((wo & bit) != 0ull) {
            dst[k] = (typename E::raw)x;
            k++;
        }
    }
}

// Pici (+) Pici -> Pici, one tile per wave and one partition per block (the
// partition's four tile counts meet in LDS, as in k_to_pici).  Each wave
// reads its tile's column words and offsets from both messages, stages both
// value ranges in its LDS buffer (one load round when together they fit
// kChunkVals, else per column group), finds exact cancellations among the
// rows both operands hold, and merges each column's two runs in row order
// into its place once the partition's offset is known by decoupled
// look-back (a minimal workspace, or a small output).  Deferred: the first
// of two passes instead -- each partition publishes its aggregate and parks
// its merged values in its own slot, as k_to_pici's first pass does (a full
// workspace below 2048 partitions; from there k_pp_part runs).
template <class E, bool Deferred>
__global__ void __launch_bounds__(kBlockThreads) k_pp_tile(PiciSinkArgs g) {
    using raw = typename E::raw;
    __shared__ raw lds_in[kWavesPerBlock][kChunkVals];
    __shared__ raw lds_out[Deferred ? kWavesPerBlock : 1][Deferred ? kChunkVals : 1];
    __shared__ uint32_t s_cnt[kWavesPerBlock];
    __shared__ uint32_t s_prefix;
    const uint32_t wave = threadIdx.x >> 6, l = lane_id();
    raw* in = lds_in[wave];
    const uint32_t p = blockIdx.x;
    const uint32_t epoch30 = g.epoch & 0x3FFFFFFFu;
    const uint64_t t = (uint64_t)p * kTilesPerPart + wave;
    const bool has_tile = t < g.T;
    const uint64_t oI = off_I(g.n), oA = off_A(g.n);
    const raw* Aa = reinterpret_cast<const raw*>(g.a.data + oA);
    const raw* Ab = reinterpret_cast<const raw*>(g.b.data + oA);

    // headers and this tile's column words / offsets first (the host
    // guarantees both capacities cover the index arrays); headers checked
    // while those are in flight
    const HeaderWords hwa = load_header_words(g.a.hdr);
    const HeaderWords hwb = load_header_words(g.b.hdr);
    const PiciMeta ma = load_pici_meta_any<E>(g.a.data, g.a.cap, t, g.n);
    const PiciMeta mb = load_pici_meta_any<E>(g.b.data, g.b.cap, t, g.n);
    const HeaderView ha = check_header(hwa, g.a.cap, g.n, E::dtype, kFmtPici);
    const HeaderView hb = check_header(hwb, g.b.cap, g.n, E::dtype, kFmtPici);
    if (!(ha.ok && hb.ok)) {          // the same in every wave: no partition publishes
        if (blockIdx.x == 0 && threadIdx.x == 0) set_status(g.ctrl, SPCCL_ERR_CORRUPT_STREAM);
        return;
    }
    PiciCols ca{0, 0, 0, 0, true}, cb{0, 0, 0, 0, true};
    uint64_t wo = 0;
    uint32_t cpo = 0, tilecnt = 0, la = 0;
    bool one = true;
    if (has_tile) {
        ca = pici_columns(ma, ha.nnz, t, g.n, g.ctrl);
        cb = pici_columns(mb, hb.nnz, t, g.n, g.ctrl);
        one = ca.cnt + cb.cnt <= kChunkVals;
        uint64_t cancel = 0;
        if (one) {
            bool zero;
            la = pp_stage<E>(ca, cb, Aa + ca.base, Ab + cb.base, 0, 64, in, zero);
            cancel = pp_cancel<E>(ca.w, cb.w, in, ca.colpref, la + cb.colpref, zero, true);
        } else {
#pragma unroll 1
            for (int h = 0; h < PPGroup::count; h++) {
                const uint32_t c0 = PPGroup::cols * h, c1 = c0 + PPGroup::cols;
                bool zg;
                const uint32_t lg = pp_stage<E>(ca, cb, Aa + ca.base, Ab + cb.base, c0, c1, in, zg);
                cancel |= pp_cancel<E>(ca.w, cb.w, in, ca.colpref - lane_bcast(ca.colpref, c0),
                                       lg + cb.colpref - lane_bcast(cb.colpref, c0), zg, l >= c0 && l < c1);
                wave_lds_sync();
            }
        }
        wo = (ca.w | cb.w) & ~cancel;
        reinterpret_cast<uint64_t*>(g.out + kHeaderBytes)[t * 64 + l] = wo;
        const uint32_t c = (uint32_t)__popcll(wo);
        cpo = wave_excl_scan(c);
        tilecnt = lane_bcast(cpo + c, 63);
    }
    if (l == 0) s_cnt[wave] = tilecnt;
    __syncthreads();
    uint32_t tile_excl = 0, agg = 0;
#pragma unroll
    for (uint32_t k = 0; k < kWavesPerBlock; k++) {
        const uint32_t ck = s_cnt[k];
        tile_excl += k < wave ? ck : 0u;
        agg += ck;
    }
    if (threadIdx.x == 0) publish(g.flags, p, epoch30, kFlagAggregate, agg);
    if constexpr (Deferred) {
        if (!has_tile) return;
        raw* slot = reinterpret_cast<raw*>(g.slots) + (uint64_t)p * kPartElems + tile_excl;
        if (one && tilecnt <= kChunkVals) {
            // merged in LDS, then to the slot with contiguous stores
            raw* ob = lds_out[Deferred ? wave : 0];
            pp_merge<E>(ca.w, cb.w, wo, in, ca.colpref, la + cb.colpref, ob, cpo, true);
            wave_lds_sync();
            for (uint32_t i = l; i < tilecnt; i += 64) slot[i] = ob[i];
        } else if (one) {
            pp_merge<E>(ca.w, cb.w, wo, in, ca.colpref, la + cb.colpref, slot, cpo, true);
        } else {
#pragma unroll 1
            for (int h = 0; h < PPGroup::count; h++) {
                const uint32_t c0 = PPGroup::cols * h, c1 = c0 + PPGroup::cols;
                bool zg;
                const uint32_t lg = pp_stage<E>(ca, cb, Aa + ca.base, Ab + cb.base, c0, c1, in, zg);
                pp_merge<E>(ca.w, cb.w, wo, in, ca.colpref - lane_bcast(ca.colpref, c0),
                            lg + cb.colpref - lane_bcast(cb.colpref, c0), slot, cpo, l >= c0 && l < c1);
                wave_lds_sync();
            }
        }
        if (l == 0) reinterpret_cast<uint32_t*>(g.out + oI)[t] = tile_excl;   // k_place adds the prefix
        return;
    }
    if (wave == 0) {
        bool ok;
        const uint32_t pre = chunk_lookback(g.flags, g.nparts, p, agg, epoch30, g.ctrl, ok);
        if (l == 0) s_prefix = ok ? pre : kNoPrefix;
    }
    __syncthreads();
    const uint32_t prefix = s_prefix;
    if (prefix == kNoPrefix) return;            // a predecessor never published: write nothing
    raw* dst = reinterpret_cast<raw*>(g.out + oA) + prefix + tile_excl;
    if (has_tile) {
        if (one) {
            pp_merge<E>(ca.w, cb.w, wo, in, ca.colpref, la + cb.colpref, dst, cpo, true);
        } else {
#pragma unroll 1
            for (int h = 0; h < PPGroup::count; h++) {
                const uint32_t c0 = PPGroup::cols * h, c1 = c0 + PPGroup::cols;
                bool zg;
                const uint32_t lg = pp_stage<E>(ca, cb, Aa + ca.base, Ab + cb.base, c0, c1, in, zg);
                pp_merge<E>(ca.w, cb.w, wo, in, ca.colpref - lane_bcast(ca.colpref, c0),
                            lg + cb.colpref - lane_bcast(cb.colpref, c0), dst, cpo, l >= c0 && l < c1);
                wave_lds_sync();
            }
        }
        if (l == 0) reinterpret_cast<uint32_t*>(g.out + oI)[t] = prefix + tile_excl;
    }
    if (p == g.nparts - 1 && threadIdx.x == 0) {
        const uint64_t nnz = (uint64_t)prefix + agg;
        uint32_t* I = reinterpret_cast<uint32_t*>(g.out + oI);
        I[g.T] = (uint32_t)nnz;
        for (uint64_t b = oI + 4 * (g.T + 1); b < oA; b += 4) *reinterpret_cast<uint32_t*>(g.out + b) = 0u;
        write_header(g.out, kFmtPici, E::dtype, g.n, nnz, oI, oA, oA + nnz * sizeof(raw));
    }
}

// Pici (+) Pici -> Pici, one partition (four tiles) per wave.  The wave
// reads the column words of its four tiles and their offsets in one round
// trip; when the partition's values (a contiguous range of each operand) fit
// the stage together, they arrive in one more; each tile's merged results go
// into an LDS output buffer in partition order, which is written to the
// partition's slot with contiguous stores whenever the next tile might not
// fit.  Tiles whose values do not fit the stage take it one tile (or one
// column group) at a time.
// Single = false: the first of two passes; the buffer goes to the slot at the
// end too, and k_place moves the slot into place (slot layout, offsets and
// counts are those k_place expects).  A wave needs no other wave.
// Single = true: the wave publishes its aggregate and finds its offset itself
// in two levels, as k_place does: the aggregates of the partitions before it
// in its chunk of kPlaceChunk, and the sum of each earlier chunk, which the
// chunk's last partition publishes (flags[P + c]) as soon as it has read its
// chunk's aggregates.  A wave waits only for lower-numbered partitions, which
// publish their aggregates before they wait for anything (and the chunk sums
// depend on nothing else), and work-groups start in index order, so every
// wait ends (bounded by the spin limit regardless).  It then moves its parked
// values and its buffer into place: no second launch, and at high sparsity
// nothing parked.
template <class E, bool Single>
__global__ void __launch_bounds__(kBlockThreads) k_pp_part(PiciSinkArgs g) {
    using raw = typename E::raw;
    constexpr int K = (int)kTilesPerPart;
    __shared__ raw lds_in[kWavesPerBlock][kChunkVals];
    __shared__ raw lds_out[kWavesPerBlock][kChunkVals];
    const uint32_t wave = threadIdx.x >> 6, l = lane_id();
    raw* in = lds_in[wave];
    raw* ob = lds_out[wave];
    const uint32_t p = blockIdx.x * kWavesPerBlock + wave;
    const uint32_t epoch30 = g.epoch & 0x3FFFFFFFu;
    const uint64_t oI = off_I(g.n), oA = off_A(g.n);
    const uint64_t t0 = (uint64_t)p * kTilesPerPart;

    // headers, the tiles' column words and offsets I[t0 .. t0 + 4] of both
    // messages, through buffer resources that end at the index arrays (the
    // host guarantees both capacities cover them; past them the hardware
    // returns zeros), so every wave issues them before any check
    const HeaderWords hwa = load_header_words(g.a.hdr);
    const HeaderWords hwb = load_header_words(g.b.hdr);
    uint64_t wa[K], wb[K];
    uint32_t Ia, Ib;                              // lane j <= 4: I[t0 + j]
    {
        const uint64_t ea = oA < g.a.cap ? oA : g.a.cap, eb = oA < g.b.cap ? oA : g.b.cap;
        const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint8_t*>(g.a.data), (short)0, (int)(uint32_t)ea, kBufferWord3);
        const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint8_t*>(g.b.data), (short)0, (int)(uint32_t)eb, kBufferWord3);
        const uint32_t tlo = __builtin_amdgcn_readfirstlane((uint32_t)t0);
#pragma unroll
        for (int k = 0; k < K; k++) {
            const uint32_t ob8 = (uint32_t)(kHeaderBytes + 512ull * (tlo + k)) + l * 8u;
            const auto x = __builtin_amdgcn_raw_buffer_load_b64(ra, ob8, 0, kStreamLoad);
            const auto y = __builtin_amdgcn_raw_buffer_load_b64(rb, ob8, 0, kStreamLoad);
            wa[k] = (uint64_t)x[0] | ((uint64_t)x[1] << 32);
            wb[k] = (uint64_t)y[0] | ((uint64_t)y[1] << 32);
        }
        const uint32_t oi = (uint32_t)(oI + 4ull * tlo) + (l <= (uint32_t)K ? 4u * l : 0u);
        Ia = __builtin_amdgcn_raw_buffer_load_b32(ra, oi, 0, kStreamLoad);
        Ib = __builtin_amdgcn_raw_buffer_load_b32(rb, oi, 0, kStreamLoad);
    }
    const HeaderView ha = check_header(hwa, g.a.cap, g.n, E::dtype, kFmtPici);
    const HeaderView hb = check_header(hwb, g.b.cap, g.n, E::dtype, kFmtPici);
    if (!(ha.ok && hb.ok)) {          // the same in every wave: no partition publishes
        if (blockIdx.x == 0 && threadIdx.x == 0) set_status(g.ctrl, SPCCL_ERR_CORRUPT_STREAM);
        return;
    }
    if (p >= g.nparts) return;
    const uint32_t ntile = g.T - t0 < (uint64_t)K ? (uint32_t)(g.T - t0) : (uint32_t)K;
    const raw* Aa = reinterpret_cast<const raw*>(g.a.data + oA);
    const raw* Ab = reinterpret_cast<const raw*>(g.b.data + oA);
    raw* slot = reinterpret_cast<raw*>(g.slots) + (uint64_t)p * kPartElems;
    uint64_t* Bo = reinterpret_cast<uint64_t*>(g.out + kHeaderBytes);

    PiciCols ca[K], cb[K];
    bool all_ok = true;
#pragma unroll
    for (int k = 0; k < K; k++) {
        if ((uint32_t)k < ntile) {
            ca[k] = pici_columns(PiciMeta{wa[k], lane_bcast(Ia, k), lane_bcast(Ia, k + 1)}, ha.nnz, t0 + k, g.n, g.ctrl);
            cb[k] = pici_columns(PiciMeta{wb[k], lane_bcast(Ib, k), lane_bcast(Ib, k + 1)}, hb.nnz, t0 + k, g.n, g.ctrl);
            all_ok = all_ok && ca[k].ok && cb[k].ok;
        } else {
            ca[k] = PiciCols{0, 0, 0, 0, true};
            cb[k] = PiciCols{0, 0, 0, 0, true};
        }
    }
    // the partition's values in one staging round when they fit together
    const uint32_t a_lo = lane_bcast(Ia, 0), b_lo = lane_bcast(Ib, 0);
    const uint32_t la = all_ok ? lane_bcast(Ia, ntile) - a_lo : 0u;
    const uint32_t lb = all_ok ? lane_bcast(Ib, ntile) - b_lo : 0u;
    const bool whole = all_ok && la + lb <= kChunkVals;
    bool zero_all = false;
    if (whole) {
        raw x[kChunkSlots];
#pragma unroll
        for (int j = 0; j < kChunkSlots; j++) {
            const uint32_t i = l + 64 * j;
            x[j] = (raw)1;
            if (stage_round<E>(j, la + lb)) x[j] = i < la ? Aa[a_lo + i] : (i < la + lb ? Ab[b_lo + (i - la)] : (raw)1);
        }
        bool z = false;
#pragma unroll
        for (int j = 0; j < kChunkSlots; j++) {
            const uint32_t i = l + 64 * j;
            if (stage_round<E>(j, la + lb)) {
                z |= x[j] == 0;
                if (i < la + lb) in[i] = x[j];
            }
        }
        zero_all = __any(z);
        wave_lds_sync();
    }

    uint32_t fill = 0, flushed = 0, excl = 0;     // values in the output buffer / written to the slot / before the tile
    uint32_t tile_rel = 0;                         // lane k < ntile: tile k's offset in the partition
    auto flush = [&]() {
        wave_lds_sync();
        for (uint32_t i = l; i < fill; i += 64) slot[flushed + i] = ob[i];
        wave_lds_sync();
        flushed += fill;
        fill = 0;
    };
    // One launch, the partition's values staged together: the four tiles'
    // counts first, published before the merges, so that the partitions after
    // this one wait less; the merged output always fits the buffer then.
    bool early = false;
    if constexpr (Single) {
        if (whole) {
            early = true;
            uint64_t wo_k[K];
            uint32_t cpo_k[K], base_k[K];
#pragma unroll
            for (int k = 0; k < K; k++) {
                wo_k[k] = 0;
                cpo_k[k] = 0;
                base_k[k] = fill;
                if ((uint32_t)k < ntile) {
                    const PiciCols& A = ca[k];
                    const PiciCols& B = cb[k];
                    const uint32_t ia = (A.base - a_lo) + A.colpref, ib = la + (B.base - b_lo) + B.colpref;
                    const uint64_t wo = (A.w | B.w) & ~pp_cancel<E>(A.w, B.w, in, ia, ib, zero_all, true);
                    Bo[(t0 + k) * 64 + l] = wo;
                    const uint32_t c = (uint32_t)__popcll(wo);
                    const uint32_t cpo = wave_excl_scan(c);
                    if (l == (uint32_t)k) tile_rel = fill;
                    fill += lane_bcast(cpo + c, 63);
                    wo_k[k] = wo;
                    cpo_k[k] = cpo;
                }
            }
            if (l == 0) publish(g.flags, p, epoch30, kFlagAggregate, fill);
#pragma unroll
            for (int k = 0; k < K; k++) {
                if ((uint32_t)k < ntile) {
                    const PiciCols& A = ca[k];
                    const PiciCols& B = cb[k];
                    pp_merge<E>(A.w, B.w, wo_k[k], in, (A.base - a_lo) + A.colpref, la + (B.base - b_lo) + B.colpref,
                                ob, base_k[k] + cpo_k[k], true);
                }
            }
        }
    }
#pragma unroll
    for (int k = 0; k < K; k++) {
        if (early || (uint32_t)k >= ntile) break;
        const PiciCols& A = ca[k];
        const PiciCols& B = cb[k];
        const uint64_t t = t0 + k;
        if (l == (uint32_t)k) tile_rel = excl;
        uint64_t cancel = 0;
        const bool one = whole || A.cnt + B.cnt <= kChunkVals;
        uint32_t ia = 0, ib = 0;
        bool zero = zero_all;
        if (whole) {
            ia = (A.base - a_lo) + A.colpref;
            ib = la + (B.base - b_lo) + B.colpref;
            cancel = pp_cancel<E>(A.w, B.w, in, ia, ib, zero, true);
        } else if (one) {
            wave_lds_sync();
            pp_stage<E>(A, B, Aa + A.base, Ab + B.base, 0, 64, in, zero);
            ia = A.colpref;
            ib = A.cnt + B.colpref;
            cancel = pp_cancel<E>(A.w, B.w, in, ia, ib, zero, true);
        } else {
#pragma unroll 1
            for (int h = 0; h < PPGroup::count; h++) {
                const uint32_t c0 = PPGroup::cols * h, c1 = c0 + PPGroup::cols;
                bool zg;
                wave_lds_sync();
                const uint32_t lg = pp_stage<E>(A, B, Aa + A.base, Ab + B.base, c0, c1, in, zg);
                cancel |= pp_cancel<E>(A.w, B.w, in, A.colpref - lane_bcast(A.colpref, c0),
                                       lg + B.colpref - lane_bcast(B.colpref, c0), zg, l >= c0 && l < c1);
            }
        }
        const uint64_t wo = (A.w | B.w) & ~cancel;
        Bo[t * 64 + l] = wo;
        const uint32_t c = (uint32_t)__popcll(wo);
        const uint32_t cpo = wave_excl_scan(c);
        const uint32_t tilecnt = lane_bcast(cpo + c, 63);
        if (one) {
            if (fill + tilecnt > kChunkVals) flush();
            pp_merge<E>(A.w, B.w, wo, in, ia, ib, ob, fill + cpo, true);
            fill += tilecnt;
        } else {
#pragma unroll 1
            for (int h = 0; h < PPGroup::count; h++) {
                const uint32_t c0 = PPGroup::cols * h, c1 = c0 + PPGroup::cols;
                const uint32_t go0 = lane_bcast(cpo, c0), go1 = c1 == 64 ? tilecnt : lane_bcast(cpo, c1);
                if (fill + (go1 - go0) > kChunkVals) flush();
                bool zg;
                wave_lds_sync();
                const uint32_t lg = pp_stage<E>(A, B, Aa + A.base, Ab + B.base, c0, c1, in, zg);
                pp_merge<E>(A.w, B.w, wo, in, A.colpref - lane_bcast(A.colpref, c0),
                            lg + B.colpref - lane_bcast(B.colpref, c0), ob, fill + cpo - go0, l >= c0 && l < c1);
                fill += go1 - go0;
            }
        }
        excl += tilecnt;
    }
    uint32_t* I = reinterpret_cast<uint32_t*>(g.out + oI);
    if constexpr (!Single) {
        flush();
        if (l < ntile) I[t0 + l] = tile_rel;       // k_place adds the prefix
        if (l == 0) publish(g.flags, p, epoch30, kFlagAggregate, flushed);
        return;
    }
    const uint32_t agg = flushed + fill;
    if (!early && l == 0) publish(g.flags, p, epoch30, kFlagAggregate, agg);
    bool ok;
    const uint32_t prefix = chunk_lookback(g.flags, g.nparts, p, agg, epoch30, g.ctrl, ok);
    if (!ok) return;                  // a predecessor never published: write nothing more
    raw* dst = reinterpret_cast<raw*>(g.out + oA) + prefix;
    if (flushed != 0) {
        __threadfence_block();        // this wave's parked values are read back below
        for (uint32_t i0 = l; i0 < flushed; i0 += 64 * 16) {
            raw x[16];
#pragma unroll
            for (int u = 0; u < 16; u++) {
                const uint32_t i = i0 + 64 * u;
                x[u] = i < flushed ? slot[i] : (raw)0;
            }
#pragma unroll
            for (int u = 0; u < 16; u++) {
                const uint32_t i = i0 + 64 * u;
                if (i < flushed) st_stream(&dst[i], x[u]);
            }
        }
    }
    wave_lds_sync();
    for (uint32_t i = l; i < fill; i += 64) st_stream(&dst[flushed + i], ob[i]);
    if (l < ntile) I[t0 + l] = prefix + tile_rel;
    if (p == g.nparts - 1 && l == 0) {
        const uint64_t nnz = (uint64_t)prefix + agg;
        I[g.T] = (uint32_t)nnz;
        for (uint64_t b = oI + 4 * (g.T + 1); b < oA; b += 4) *reinterpret_cast<uint32_t*>(g.out + b) = 0u;
        write_header(g.out, kFmtPici, E::dtype, g.n, nnz, oI, oA, oA + nnz * sizeof(raw));
    }
}

// Second pass of the two-pass Pici sink.  Every aggregate is final when this
// kernel starts (the first pass has completed), so a partition's offset is a
// sum of final numbers, found in two levels instead of by adding up all p
// predecessors (p loads for partition p, O(P^2) for the pass): the partitions
// are grouped in chunks of kPlaceChunk, block c of the first
// num_place_chunks(P) blocks adds up chunk c's aggregates and publishes the
// sum in the look-back word that follows the partitions' (flags[P + c]), and
// a block adds the sums of the chunks before its own to the aggregates of
// its own chunk's partitions before it.  A block waits only for chunk sums
// published by lower-numbered blocks, which publish before they wait for
// anything, and work-groups start in index order, so every wait ends (a spin
// limit bounds it regardless and turns a stall into SPCCL_ERR_TIMEOUT).
constexpr uint32_t kNoAggregate = 0xFFFFFFFFu;   // a partition the first pass did not publish
constexpr uint32_t kPlacePer = kWavesPerBlock;   // partitions placed by one block (one per wave)
static_assert(kPlaceChunk == kBlockThreads, "one aggregate of a chunk per thread");
static_assert(kPlaceChunk % kPlacePer == 0, "a block's partitions lie in one chunk");

// Each wave moves one partition.  Its own aggregate, the first kEarly slot
// values per lane, its tiles' relative offsets and one aggregate per thread
// (its chunk's predecessors and, for a summing block, the chunk it sums) are
// read at once; once the aggregate is known the rest of the partition's values
// (up to kMore per lane) are read while the block waits for the chunk sums;
// then every store.  Reads waited for after a store would also wait for that
// store, hence all reads first.
template <class E>
__device__ __forceinline__ void place_body(const PiciSinkArgs& g) {
    using raw = typename E::raw;
    constexpr uint32_t kEarly = 4;          // slot values per lane read before the aggregate is known
    constexpr uint32_t kMore = 16;          // slot values per lane read once it is
    __shared__ uint32_t s_base, s_part[kWavesPerBlock], s_csum[kWavesPerBlock], s_agg[kPlacePer];
    __shared__ bool s_ok;
    const uint32_t wave = threadIdx.x >> 6, l = lane_id();
    const uint32_t p0 = blockIdx.x * kPlacePer;
    const uint32_t p = p0 + wave;
    const bool mine = p < g.nparts;
    const uint32_t epoch30 = g.epoch & 0x3FFFFFFFu;
    const uint64_t oI = off_I(g.n), oA = off_A(g.n);
    uint32_t* I = reinterpret_cast<uint32_t*>(g.out + oI);
    const raw* slot = reinterpret_cast<const raw*>(g.slots) + (uint64_t)p * kPartElems;
    uint64_t* csums = g.flags + g.nparts;
    const uint32_t chunk = p0 / kPlaceChunk;
    const bool summer = blockIdx.x < num_place_chunks(g.nparts);

    // independent of every offset: own aggregate word, first slot values
    // (a slot always has kPartElems of room), the tiles' relative offsets,
    // the aggregates this block adds up
    const uint64_t f = mine ? g.flags[p] : 0ull;
    raw early[kEarly];
#pragma unroll
    for (uint32_t u = 0; u < kEarly; u++) early[u] = mine ? slot[l + 64 * u] : (raw)0;
    const uint64_t t = (uint64_t)p * kTilesPerPart + l;
    const uint32_t tile_rel = (mine && l < kTilesPerPart && t < g.T) ? I[t] : 0u;
    const uint32_t qp = chunk * kPlaceChunk + threadIdx.x;           // a predecessor in this chunk
    uint32_t part = qp < p0 ? (uint32_t)g.flags[qp] : 0u;
    const uint32_t qs = blockIdx.x * kPlaceChunk + threadIdx.x;      // a partition of the summed chunk
    uint32_t csum = 0;
    if (summer && qs < g.nparts) {
        const uint64_t fs = g.flags[qs];
        csum = (uint32_t)(fs >> 34) == epoch30 ? (uint32_t)fs : 0u;
    }
    uint32_t agg = (uint32_t)f;
    bool bad = mine && ((uint32_t)(f >> 34) != epoch30 || agg > kPartElems);   // the first pass did not run
    if (bad) agg = 0;
    if (!mine) agg = 0;
    raw more[kMore];
#pragma unroll
    for (uint32_t u = 0; u < kMore; u++) {
        const uint32_t i = l + 64 * (kEarly + u);
        more[u] = i < agg ? slot[i] : (raw)0;
    }
    part = wave_sum(part);
    csum = wave_sum(csum);
    if (l == 0) {
        s_part[wave] = part;
        s_csum[wave] = csum;
        s_agg[wave] = bad ? kNoAggregate : agg;
        if (bad) set_status(g.ctrl, SPCCL_ERR_WORKSPACE);
    }
    __syncthreads();
    if (summer && threadIdx.x == 0) {
        uint32_t sum = 0;
#pragma unroll
        for (uint32_t k = 0; k < kWavesPerBlock; k++) sum += s_csum[k];
        publish(g.flags, g.nparts + blockIdx.x, epoch30, kFlagPrefix, sum);
    }
    bool any_bad = false;
    uint32_t prefix = 0;
#pragma unroll
    for (uint32_t k = 0; k < kPlacePer; k++) {
        const uint32_t ak = s_agg[k];
        any_bad = any_bad || ak == kNoAggregate;
        prefix += k < wave ? ak : 0u;
    }
    if (any_bad) return;          // the first pass stopped at a bad header: write nothing
#pragma unroll
    for (uint32_t k = 0; k < kWavesPerBlock; k++) prefix += s_part[k];
    if (chunk != 0) {
        // the sums of chunks 0 .. chunk-1, 64 per round, each round until
        // every one of them carries this call's epoch
        if (wave == 0) {
            uint32_t sum = 0;
            bool ok = true;
            for (uint32_t k0 = 0; k0 < chunk && ok; k0 += 64) {
                const uint32_t k = k0 + l;
                uint64_t fk = 0;
                bool ready = k >= chunk;
                uint32_t spins = 0;
                while (true) {
                    if (!ready) {
                        fk = __hip_atomic_load(&csums[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        ready = (uint32_t)(fk >> 34) == epoch30;
                    }
                    if (__all(ready)) break;
                    if (++spins > kSpinLimit) {
                        if (l == 0) set_status(g.ctrl, SPCCL_ERR_TIMEOUT);
                        ok = false;
                        break;
                    }
                    __builtin_amdgcn_s_sleep(1);
                }
                sum += k < chunk ? (uint32_t)fk : 0u;
            }
            sum = wave_sum(sum);
            if (l == 0) {
                s_base = sum;
                s_ok = ok;
            }
        }
        __syncthreads();
        if (!s_ok) return;        // a chunk sum never came: write nothing
        prefix += s_base;
    }
    if (!mine) return;
    raw* dst = reinterpret_cast<raw*>(g.out + oA) + prefix;
#pragma unroll
    for (uint32_t u = 0; u < kEarly; u++) {
        const uint32_t i = l + 64 * u;
        if (i < agg) st_stream(&dst[i], early[u]);
    }
#pragma unroll
    for (uint32_t u = 0; u < kMore; u++) {
        const uint32_t i = l + 64 * (kEarly + u);
        if (i < agg) st_stream(&dst[i], more[u]);
    }
    for (uint32_t i0 = l + 64 * (kEarly + kMore); i0 < agg; i0 += 64 * 16) {
        raw x[16];
#pragma unroll
        for (int u = 0; u < 16; u++) {
            const uint32_t i = i0 + 64 * u;
            x[u] = i < agg ? slot[i] : (raw)0;
        }
#pragma unroll
        for (int u = 0; u < 16; u++) {
            const uint32_t i = i0 + 64 * u;
            if (i < agg) st_stream(&dst[i], x[u]);
        }
    }
    if (l < kTilesPerPart && t < g.T) I[t] = tile_rel + prefix;
    if (p == g.nparts - 1 && l == 0) {
        const uint64_t nnz = (uint64_t)prefix + agg;
        I[g.T] = (uint32_t)nnz;
        for (uint64_t b = oI + 4 * (g.T + 1); b < oA; b += 4) *reinterpret_cast<uint32_t*>(g.out + b) = 0u;
        write_header(g.out, kFmtPici, E::dtype, g.n, nnz, oI, oA, oA + nnz * sizeof(raw));
    }
}

template <class E>
__global__ void __launch_bounds__(kBlockThreads) k_place(PiciSinkArgs g) {
    place_body<E>(g);
}

template <class E>
__global__ void __launch_bounds__(kBlockThreads) k_place_rb(PiciSinkArgs g, RankBatch rb) {
    if (rank_skipped(rb, blockIdx.y)) return;
    place_body<E>(rank_sink(g, rb, blockIdx.y));
}

// ---------------------------------------------------------------------------
// Tile index of a COO message: idx[t] = epoch << 32 | the first entry whose
// index is >= 4096 t, for t = 0 .. T (idx[T] = nnz).  One thread per entry i
// (and one for the end, i = nnz) writes the tiles between its predecessor's
// tile and its own -- at most the last kIdxSpan of them, so a corrupt J that
// jumps back and forth cannot make a thread write the whole index -- and the
// index is read in one pass over J.  Tiles left unwritten keep words of an
// earlier epoch (or none) and search J instead, so the index only ever saves
// work: in a valid message every written word is exact.  Entries that are not
// strictly increasing or not below n are flagged (the tiles check their
// entries again as they use them).
constexpr uint64_t kIdxSpan = 64;

__global__ void __launch_bounds__(256) k_coo_index(const uint8_t* msg, uint64_t cap, uint64_t n, int dtype,
                                                  uint64_t* idx, uint32_t epoch, WsCtrl* ctrl) {
    const HeaderView h = read_header(msg, cap, n, dtype, kFmtCoo);
    if (!h.ok) {
        if (blockIdx.x == 0 && threadIdx.x == 0) set_status(ctrl, SPCCL_ERR_CORRUPT_STREAM);
        return;
    }
    const uint64_t T = num_tiles(n), nnz = h.nnz;
    const uint64_t tag = (uint64_t)epoch << 32;
    const uint32_t* J = reinterpret_cast<const uint32_t*>(msg + kHeaderBytes);
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i <= nnz;
         i += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t cur = i < nnz ? J[i] : n;
        const uint64_t prev = i > 0 ? J[i - 1] : 0;
        if (i < nnz && (cur >= n || (i > 0 && cur <= prev))) set_status(ctrl, SPCCL_ERR_CORRUPT_STREAM);
        // tiles (tile(prev), tile(cur)] start at entry i (all of [0, tile(cur)] for the first)
        uint64_t first = i > 0 ? prev / kTileElems + 1 : 0;
        uint64_t last = i < nnz ? cur / kTileElems : T;
        if (last > T) last = T;
        if (last >= kIdxSpan && first < last - kIdxSpan + 1) first = last - kIdxSpan + 1;
        for (uint64_t t = first; t <= last; t++) idx[t] = tag | i;
    }
}

// ---------------------------------------------------------------------------
// COO sink: out = COO(srcA (+) srcB) (Sec. II-B format), in two passes.
// The value array of a COO message starts after all nnz indices, so no entry
// can be placed before the total is known:
//   k_to_coo       each partition (one block, one tile per wave) computes its
//                  tiles, counts, publishes its aggregate and parks its
//                  (index, value) entries in its own worst-case slots; never
//                  waits on another block;
//   k_place_coo    the partitions' offsets and the total from per-chunk sums
//                  of the aggregates, the header and the pad; one wave per
//                  partition moves its entries into place.
// Entries leave a tile in row-major order, i.e. by increasing flat index:
// row r's present lanes are a ballot mask, and each takes the position of
// the set bits below it.

constexpr uint32_t kCooOut = 1024;             // entries staged per wave before a flush

template <class E, int SA, int SB>
__global__ void __launch_bounds__(kBlockThreads) k_to_coo(PiciSinkArgs g) {
    using raw = typename E::raw;
    constexpr bool coo_in = SA == SRC_COO || SB == SRC_COO;
    __shared__ raw stage_all[kWavesPerBlock][kCooOut * 4 / sizeof(raw)];   // input chunks, then output values
    __shared__ uint32_t sidx_all[kWavesPerBlock][kCooOut];
    __shared__ CooLds coo_all[coo_in ? kWavesPerBlock : 1];
    __shared__ uint32_t s_cnt[kWavesPerBlock];
    const uint32_t wave = threadIdx.x >> 6, l = lane_id();
    raw* stage = stage_all[wave];
    uint32_t* sidx = sidx_all[wave];
    const uint32_t p = blockIdx.x;
    const uint32_t epoch30 = g.epoch & 0x3FFFFFFFu;
    const uint64_t t = (uint64_t)p * kTilesPerPart + wave;
    const bool has_tile = t < g.T;
    uint32_t v[64];
    if (!load_tile_pair<E, SA, SB>(g.a, g.b, t, has_tile, g.n, stage, &coo_all[coo_in ? wave : 0], g.ctrl, v))
        return;                   // uniform over the grid: no partition publishes
    uint32_t tilecnt = 0;
    if (has_tile) {
#pragma unroll
        for (int r = 0; r < 64; r++) tilecnt += (uint32_t)__popcll(__ballot(v[r] != 0u));
    }
    if (l == 0) s_cnt[wave] = tilecnt;
    __syncthreads();
    uint32_t tile_excl = 0, agg = 0;
#pragma unroll
    for (uint32_t k = 0; k < kWavesPerBlock; k++) {
        const uint32_t ck = s_cnt[k];
        tile_excl += k < wave ? ck : 0u;
        agg += ck;
    }
    if (threadIdx.x == 0) publish(g.flags, p, epoch30, kFlagAggregate, agg);
    if (!has_tile) return;
    uint32_t* islot = g.idx_slots + (uint64_t)p * kPartElems + tile_excl;
    raw* vslot = reinterpret_cast<raw*>(g.slots) + (uint64_t)p * kPartElems + tile_excl;
    const uint32_t base_idx = (uint32_t)(t * kTileElems) + l;
    uint32_t done = 0, rank = 0;                 // entries flushed, entries staged
    wave_lds_sync();                             // the COO source's stage reads are over
#pragma unroll
    for (int r = 0; r < 64; r++) {
        const uint64_t m = __ballot(v[r] != 0u);
        if (m) {
            const uint32_t c = (uint32_t)__popcll(m);
            if (rank + c > kCooOut) {
                wave_lds_sync();
                for (uint32_t i = l; i < rank; i += 64) { islot[done + i] = sidx[i]; vslot[done + i] = stage[i]; }
                wave_lds_sync();
                done += rank;
                rank = 0;
            }
            if (v[r] != 0u) {
                const uint32_t pos = rank + bits_below_lane(m);
                sidx[pos] = base_idx + 64u * (uint32_t)r;
                stage[pos] = (raw)v[r];
            }
            rank += c;
        }
    }
    wave_lds_sync();
    for (uint32_t i = l; i < rank; i += 64) { islot[done + i] = sidx[i]; vslot[done + i] = stage[i]; }
}

// Second pass of the COO sink, one wave per partition.  The values' offset
// depends on the total count, so every block needs every partition's
// aggregate: as in the Pici place pass, block c of the first
// num_place_chunks(P) blocks adds up chunk c's aggregates and publishes the
// sum (flags[P + c]; state kFlagAggregate instead of kFlagPrefix if a
// partition of the chunk did not publish: an input failed its header check
// and nothing is written), and every block adds the chunk sums up to its
// prefix and to the total.  The summing blocks publish before they wait for
// anything and are the lowest-numbered ones, which start first and all fit
// the device at once (at most 1024 blocks for n < 2^32), so every wait ends;
// a spin limit bounds it regardless and turns a stall into SPCCL_ERR_TIMEOUT.
// Block 0 writes the header and the pad between J and V.
template <class E>
__global__ void __launch_bounds__(kBlockThreads) k_place_coo(PiciSinkArgs g) {
    using raw = typename E::raw;
    constexpr int U = 8;
    __shared__ uint32_t s_part[kWavesPerBlock], s_csum[kWavesPerBlock], s_bad[kWavesPerBlock], s_agg[kWavesPerBlock];
    __shared__ uint32_t s_base, s_total, s_ok;
    const uint32_t wave = threadIdx.x >> 6, l = lane_id();
    const uint32_t p0 = blockIdx.x * kWavesPerBlock;
    const uint32_t p = p0 + wave;
    const bool mine = p < g.nparts;
    const uint32_t epoch30 = g.epoch & 0x3FFFFFFFu;
    const uint32_t nchunks = (uint32_t)num_place_chunks(g.nparts);
    const uint32_t chunk = p0 / kPlaceChunk;
    const bool summer = blockIdx.x < nchunks;
    uint64_t* csums = g.flags + g.nparts;

    const uint64_t f = mine ? g.flags[p] : 0ull;
    const uint32_t qp = chunk * kPlaceChunk + threadIdx.x;           // a predecessor in this chunk
    uint32_t part = qp < p0 ? (uint32_t)g.flags[qp] : 0u;
    const uint32_t qs = blockIdx.x * kPlaceChunk + threadIdx.x;      // a partition of the summed chunk
    uint32_t csum = 0, bad = 0;
    if (summer && qs < g.nparts) {
        const uint64_t fs = g.flags[qs];
        bad = (uint32_t)(fs >> 34) != epoch30 || (uint32_t)fs > kPartElems;
        csum = bad ? 0u : (uint32_t)fs;
    }
    part = wave_sum(part);
    csum = wave_sum(csum);
    bad = wave_or(bad);
    if (l == 0) {
        s_part[wave] = part;
        s_csum[wave] = csum;
        s_bad[wave] = bad;
        s_agg[wave] = mine ? (uint32_t)f : 0u;
    }
    __syncthreads();
    if (summer && threadIdx.x == 0) {
        uint32_t sum = 0, any = 0;
#pragma unroll
        for (uint32_t k = 0; k < kWavesPerBlock; k++) { sum += s_csum[k]; any |= s_bad[k]; }
        if (any) set_status(g.ctrl, SPCCL_ERR_WORKSPACE);
        publish(g.flags, g.nparts + blockIdx.x, epoch30, any ? kFlagAggregate : kFlagPrefix, sum);
    }
    // every chunk sum, 64 per round, each round until all carry this call's epoch
    if (wave == 0) {
        uint32_t before = 0, total = 0;
        bool ok = true;
        for (uint32_t k0 = 0; k0 < nchunks && ok; k0 += 64) {
            const uint32_t k = k0 + l;
            uint64_t fk = 0;
            bool ready = k >= nchunks;
            uint32_t spins = 0;
            while (true) {
                if (!ready) {
                    fk = __hip_atomic_load(&csums[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    ready = (uint32_t)(fk >> 34) == epoch30;
                }
                if (__all(ready)) break;
                if (++spins > kSpinLimit) {
                    if (l == 0) set_status(g.ctrl, SPCCL_ERR_TIMEOUT);
                    ok = false;
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
            ok = ok && !__any(k < nchunks && ((uint32_t)(fk >> 32) & 3u) != kFlagPrefix);
            const uint32_t v = k < nchunks ? (uint32_t)fk : 0u;
            before += wave_sum(k < chunk ? v : 0u);
            total += wave_sum(v);
        }
        if (l == 0) {
            s_base = before;
            s_total = total;
            s_ok = ok;
        }
    }
    __syncthreads();
    if (!s_ok) return;            // a partition did not publish, or a chunk sum never came: write nothing
    uint32_t prefix = s_base;
#pragma unroll
    for (uint32_t k = 0; k < kWavesPerBlock; k++) prefix += s_part[k] + (k < wave ? s_agg[k] : 0u);
    const uint64_t nnz = s_total, oV = coo_off_V(nnz);
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        write_header(g.out, kFmtCoo, E::dtype, g.n, nnz, kHeaderBytes, oV, coo_bytes(E::dtype, nnz));
        for (uint64_t b = kHeaderBytes + 4 * nnz; b < oV; b++) g.out[b] = 0;
    }
    if (!mine) return;
    const uint32_t cnt = (uint32_t)f;
    const uint32_t* islot = g.idx_slots + (uint64_t)p * kPartElems;
    const raw* vslot = reinterpret_cast<const raw*>(g.slots) + (uint64_t)p * kPartElems;
    uint32_t* J = reinterpret_cast<uint32_t*>(g.out + kHeaderBytes) + prefix;
    raw* V = reinterpret_cast<raw*>(g.out + oV) + prefix;
    for (uint32_t i0 = l; i0 < cnt; i0 += 64 * U) {
        uint32_t x[U];
        raw y[U];
#pragma unroll
        for (int u = 0; u < U; u++) {
            const uint32_t i = i0 + 64 * u;
            x[u] = i < cnt ? islot[i] : 0u;
            y[u] = i < cnt ? vslot[i] : (raw)0;
        }
#pragma unroll
        for (int u = 0; u < U; u++) {
            const uint32_t i = i0 + 64 * u;
            if (i < cnt) { J[i] = x[u]; V[i] = y[u]; }
        }
    }
}

// ---------------------------------------------------------------------------
// Dense sink: out[i] = (srcA (+) srcB)[i] for every i < n.

template <class E>
__device__ __forceinline__ void store_tile(uint8_t* out, uint64_t t, uint64_t n, const uint32_t (&v)[64]) {
    using raw = typename E::raw;
    const uint32_t l = lane_id();
    raw* col = reinterpret_cast<raw*>(out) + t * kTileElems + l;
    const uint64_t rem = n - t * kTileElems;
    if (rem >= kTileElems) {
#pragma unroll
        for (int r = 0; r < 64; r++) st_stream(&col[64 * r], (raw)v[r]);
    } else {
#pragma unroll
        for (int r = 0; r < 64; r++)
            if ((uint64_t)(64 * r + l) < rem) st_stream(&col[64 * r], (raw)v[r]);
    }
}

template <class E, int SA, int SB>
__device__ __forceinline__ void to_dense_body(const DenseSinkArgs& g) {
    using raw = typename E::raw;
    constexpr bool coo = SA == SRC_COO || SB == SRC_COO;
    __shared__ raw stage_all[kWavesPerBlock][E::cap];
    __shared__ CooLds coo_all[coo ? kWavesPerBlock : 1];
    const uint32_t wave = threadIdx.x >> 6;
    const uint64_t t = (uint64_t)blockIdx.x * kWavesPerBlock + wave;
    const bool has_tile = t < g.T;
    uint32_t v[64];
    raw* col = (has_tile && g.n - t * kTileElems >= kTileElems)
                   ? reinterpret_cast<raw*>(g.out) + t * kTileElems + lane_id() : nullptr;
    bool stored = false;
    if (!load_tile_pair<E, SA, SB>(g.a, g.b, t, has_tile, g.n, stage_all[wave], &coo_all[coo ? wave : 0], g.ctrl, v,
                                   col, &stored))
        return;
    if (blockIdx.x == 0 && threadIdx.x == 0 && g.out_hdr)
        write_header(g.out_hdr, kFmtDense, E::dtype, g.n, kNnzUnknown, 0, kHeaderBytes, dense_msg_bytes(g.n, E::dtype));
    if (!has_tile || stored) return;
    store_tile<E>(g.out, t, g.n, v);
}

template <class E, int SA, int SB>
__global__ void __launch_bounds__(kBlockThreads) k_to_dense(DenseSinkArgs g) {
    to_dense_body<E, SA, SB>(g);
}

template <class E, int SA, int SB>
__global__ void __launch_bounds__(kBlockThreads) k_to_dense_rb(DenseSinkArgs g, RankBatch rb) {
    if (rank_skipped(rb, blockIdx.y)) return;
    to_dense_body<E, SA, SB>(rank_dense(g, rb, blockIdx.y));
}

// Expansion of P parts (all-gather receive side and decompress): the format
// of each message (dense, Pici or COO) is read from its header on the
// device.
//
// Each wave expands K consecutive tiles of one part and issues its reads
// before its first store: the K tiles' column words and offsets, then, in one
// go, the values of as many leading tiles as fit kChunkVals (their value
// ranges are contiguous), held in registers and staged in LDS; then it writes
// the dense tiles.  On this architecture one counter tracks both loads and
// stores, so a read that has to be waited for after a store also waits for
// that store; with the reads in front the writes stream and the read latency
// is paid once per K tiles.  Tiles that do not fit are expanded one at a
// time (stage their values, then write), and a tile holding more than
// kChunkVals values reads its column runs per lane, 16 rows at a time.
// Rows [r0, r0 + 16) of dense tile t (bounded buffer loads, zero past n).
template <class E>
__device__ __forceinline__ void fetch_dense_rows16(const uint8_t* base, uint64_t t, uint64_t n, int r0,
                                                   uint32_t (&v)[16]) {
    using raw = typename E::raw;
    constexpr uint32_t rowb = 64 * sizeof(raw);
    t = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(t >> 32)) << 32) |
        __builtin_amdgcn_readfirstlane((uint32_t)t);
    const uint64_t start = t * kTileElems;
    const uint64_t rem = start < n ? n - start : 0;
    const uint32_t bytes = (uint32_t)((rem < kTileElems ? rem : kTileElems) * sizeof(raw));
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(base) + (rem ? start : 0) * sizeof(raw), (short)0, (int)bytes, kBufferWord3);
    const uint32_t lo = lane_id() * (uint32_t)sizeof(raw);
    const int soff = (int)(rowb * (uint32_t)r0);
#pragma unroll
    for (int q = 0; q < 16; q++) {
        if constexpr (sizeof(raw) == 4)
            v[q] = __builtin_amdgcn_raw_buffer_load_b32(rs, lo + rowb * q, soff, kStreamLoad);
        else
            v[q] = __builtin_amdgcn_raw_buffer_load_b16(rs, lo + rowb * q, soff, kStreamLoad);
    }
}

// One tile from the LDS stage: value of row r of this lane's column is
// stage[rank] for its set bits, rank counting up from `rank`.  bf16 rows go
// out with streaming stores (2.2 us faster over a 256 MiB decompress), fp32
// rows with ordinary ones (1.5 us faster than streaming there).
template <class E>
__device__ __forceinline__ void store_row(typename E::raw* p, typename E::raw v) {
    if constexpr (sizeof(typename E::raw) == 2) st_stream(p, v);
    else *p = v;
}

template <class E>
__device__ __forceinline__ void store_from_stage(typename E::raw* col, uint64_t rem, uint64_t w,
                                                 const typename E::raw* stage, uint32_t rank) {
    using raw = typename E::raw;
    const uint32_t l = lane_id();
    if (rem >= kTileElems) {
#pragma unroll 8
        for (int r = 0; r < 64; r++) {
            raw v = 0;
            if ((w >> r) & 1ull) { v = stage[rank]; rank++; }
            store_row<E>(&col[64 * r], v);
        }
    } else {
#pragma unroll 8
        for (int r = 0; r < 64; r++) {
            raw v = 0;
            if ((w >> r) & 1ull) { v = stage[rank]; rank++; }
            if ((uint64_t)(64 * r + l) < rem) store_row<E>(&col[64 * r], v);
        }
    }
}

// Tiles [t0, tend) of a COO expansion, from entries lo .. lo + cnt of J and
// V (checked, in index order), a quarter tile (16 rows, kChunkVals elements)
// at a time: the quarter is zeroed in the wave's LDS buffer, the entries that
// fall in it are written there, and it is stored with 16-byte stores (element
// stores when out is not 16-byte aligned).  Entries are held in registers a
// chunk (kCooChunk) at a time, the first chunk (m entries) already loaded; a
// quarter takes entries from the next chunks until the held chunk reaches
// past it.  Every element is written once: zeroing the output first and then
// storing the values over it wrote the lines twice.  Elements at or past n are
// not written.
template <class E>
__device__ __forceinline__ void coo_tiles_lds(const uint32_t* J, const typename E::raw* V, uint32_t lo, uint32_t cnt,
                                              uint32_t m, uint32_t (&x)[kCooSlots], typename E::raw (&val)[kCooSlots],
                                              uint64_t t0, uint64_t tend, uint64_t n, typename E::raw* out,
                                              typename E::raw* buf) {
    using raw = typename E::raw;
    constexpr uint32_t per16 = 16 / sizeof(raw);
    constexpr uint32_t chunks = kChunkVals / per16;           // 16-byte chunks of a quarter
    static_assert(chunks % 64 == 0, "whole chunks per lane");
    const uint32_t l = lane_id();
    const bool vec = (reinterpret_cast<uintptr_t>(out) & 15u) == 0;
    uint4* b4 = reinterpret_cast<uint4*>(buf);
    uint32_t c0 = 0;                                          // entries before the held chunk
#pragma unroll 1
    for (uint64_t base = t0 * kTileElems; base < tend * kTileElems && base < n; base += kChunkVals) {
        const uint64_t rem = n - base;
        const uint32_t b32 = (uint32_t)base;                  // indices are below 2^32
#pragma unroll
        for (uint32_t k = 0; k < chunks / 64; k++) b4[l + 64 * k] = uint4{0, 0, 0, 0};
        wave_lds_sync();
#pragma unroll 1
        while (true) {
#pragma unroll
            for (int q = 0; q < kCooSlots; q++) {
                const uint32_t rel = x[q] - b32;
                if (l + 64u * q < m && rel < kChunkVals) buf[rel] = val[q];
            }
            if (c0 + m >= cnt) break;                         // no entries beyond the held chunk
            uint32_t xl = 0;                                  // index of the held chunk's last entry
#pragma unroll
            for (int q = 0; q < kCooSlots; q++)
                if ((uint32_t)q == (m - 1) / 64) xl = x[q];
            if (lane_bcast(xl, (m - 1) % 64) - b32 >= kChunkVals) break;   // it reaches past this quarter
            c0 += m;
            m = cnt - c0 < kCooChunk ? cnt - c0 : kCooChunk;
            coo_load_pairs<E>(J, V, lo + c0, m, false, 0, 0, x, val);
        }
        wave_lds_sync();
        raw* o = out + base;
#pragma unroll
        for (uint32_t k = 0; k < chunks / 64; k++) {
            const uint32_t c = l + 64 * k;
            const uint64_t e0 = (uint64_t)c * per16;
            if (vec && e0 + per16 <= rem) {
                st_stream(reinterpret_cast<uint4*>(o) + c, b4[c]);
            } else if (e0 < rem) {
                const uint32_t k1 = rem - e0 < per16 ? (uint32_t)(rem - e0) : per16;
                for (uint32_t k = 0; k < k1; k++) st_stream(&o[e0 + k], buf[e0 + k]);
            }
        }
        wave_lds_sync();
    }
}

// Tiles [t0, t0 + K) of one checked message (format fmt, nnz nonzeros, n
// elements, T tiles; d = its dense values for a dense message, msg = the
// message for a Pici one) expanded into out[0 .. n).  One wave; all reads
// before the first store (see k_gather).
template <class E, int K>
__device__ __forceinline__ void expand_tiles(const uint8_t* msg, const uint8_t* d, uint32_t fmt, uint64_t nnz,
                                             uint64_t n, uint64_t T, uint64_t t0, typename E::raw* out,
                                             typename E::raw* stage, WsCtrl* ctrl) {
    using raw = typename E::raw;
    const uint32_t l = lane_id();
    const uint64_t g_n = n, g_T = T;
    if (fmt == (uint32_t)kFmtCoo) {
        // The wave's entry range, searched over the whole index array (so
        // neighbouring waves meet exactly), its entries checked (inside the
        // wave's tiles, below n, strictly increasing: as they are loaded when
        // they fit one chunk, else in a pass of their own first), then the
        // tiles assembled in LDS a quarter at a time (coo_tiles_lds).
        const uint32_t* J = reinterpret_cast<const uint32_t*>(msg + kHeaderBytes);
        const raw* V = reinterpret_cast<const raw*>(msg + coo_off_V(nnz));
        const uint64_t tend = t0 + K < g_T ? t0 + K : g_T;
        const uint64_t first = t0 * kTileElems, limit = tend * kTileElems < g_n ? tend * kTileElems : g_n;
        const uint32_t b = coo_lower_bound<2>(J, 0u, (uint32_t)nnz, (l < 32 ? t0 : tend) * kTileElems);
        const uint32_t lo = lane_bcast(b, 0), hi = lane_bcast(b, 32);
        bool ok = hi >= lo && hi - lo <= (uint32_t)(tend - t0) * kTileElems && (tend < g_T || hi == nnz);
        const bool one = ok && hi - lo <= kCooChunk;
        if (ok && !one) ok = coo_span_ok(J, lo, hi, first, limit);
        uint32_t cnt = ok ? hi - lo : 0u;
        uint32_t x[kCooSlots];
        raw val[kCooSlots];
        uint32_t m = cnt < kCooChunk ? cnt : kCooChunk;
        if (m) ok = coo_load_pairs<E>(J, V, lo, m, one, first, limit, x, val);
        if (!ok) {
            cnt = m = 0;
            if (l == 0) set_status(ctrl, SPCCL_ERR_CORRUPT_STREAM);
        }
        coo_tiles_lds<E>(J, V, lo, cnt, m, x, val, t0, tend, g_n, out, stage);
        return;
    }
    if (fmt != (uint32_t)kFmtPici) {
        // a dense message: a plain copy of the wave's tiles, 16 bytes per
        // lane with eight loads in flight before their stores when source
        // and destination are 16-byte aligned (4.7 -> 6 TB/s for the dense
        // parts of an all-gather hop); else 16 rows at a time
        if (((reinterpret_cast<uintptr_t>(d) | reinterpret_cast<uintptr_t>(out)) & 15u) == 0) {
            const uint64_t e_lo = t0 * kTileElems;
            const uint64_t e_hi = (t0 + K) * kTileElems < g_n ? (t0 + K) * kTileElems : g_n;
            const uint64_t nv = (e_hi - e_lo) * sizeof(raw) / 16;
            const u32x4* s4 = reinterpret_cast<const u32x4*>(reinterpret_cast<const raw*>(d) + e_lo);
            u32x4* d4 = reinterpret_cast<u32x4*>(out + e_lo);
#pragma unroll 1
            for (uint64_t i0 = l; i0 < nv; i0 += 64 * 8) {
                u32x4 x[8];
#pragma unroll
                for (int u = 0; u < 8; u++)
                    x[u] = i0 + 64u * u < nv ? __builtin_nontemporal_load(&s4[i0 + 64u * u]) : u32x4{0, 0, 0, 0};
#pragma unroll
                for (int u = 0; u < 8; u++)
                    if (i0 + 64u * u < nv) __builtin_nontemporal_store(x[u], &d4[i0 + 64u * u]);
            }
            const raw* se = reinterpret_cast<const raw*>(d);
            for (uint64_t e = e_lo + nv * 16 / sizeof(raw) + l; e < e_hi; e += 64) out[e] = se[e];
            return;
        }
#pragma unroll 1
        for (int k = 0; k < K; k++) {
            const uint64_t t = t0 + k;
            if (t >= g_T) break;
            raw* col = out + t * kTileElems + l;
            const uint64_t rem = g_n - t * kTileElems;
#pragma unroll 1
            for (int h = 0; h < 4; h++) {
                uint32_t v[16];
                fetch_dense_rows16<E>(d, t, g_n, 16 * h, v);
#pragma unroll
                for (int q = 0; q < 16; q++) {
                    const int r = 16 * h + q;
                    if ((uint64_t)(64 * r + l) < rem) st_stream(&col[64 * r], (raw)v[q]);
                }
            }
        }
        return;
    }
    const raw* A = reinterpret_cast<const raw*>(msg + off_A(g_n));
    PiciMeta m[K];
#pragma unroll
    for (int k = 0; k < K; k++)
        m[k] = t0 + k < g_T ? load_pici_meta<E>(msg, t0 + k, g_n) : PiciMeta{0, 0, 0};
    uint64_t cw[K];
    uint32_t cpref[K], ccnt[K], cbase[K];
    int kfit = 0;                       // leading tiles whose values are staged together
#pragma unroll
    for (int k = 0; k < K; k++) {
        const bool have = t0 + k < g_T;
        const PiciCols c = have ? pici_columns(m[k], nnz, t0 + k, g_n, ctrl) : PiciCols{0, 0, 0, 0, false};
        cw[k] = c.w; cpref[k] = c.colpref; ccnt[k] = c.cnt; cbase[k] = c.base;
        // valid tiles chain (base + cnt == next == the next tile's base)
        if (kfit == k && c.ok && (c.base - cbase[0]) + c.cnt <= kChunkVals) kfit = k + 1;
    }
    const uint32_t chunk = kfit ? (cbase[kfit - 1] - cbase[0]) + ccnt[kfit - 1] : 0u;
    {
        uint32_t x[kChunkSlots];
#pragma unroll
        for (int j = 0; j < kChunkSlots; j++) {
            const uint32_t i = l + 64 * j;
            x[j] = i < chunk ? (uint32_t)A[cbase[0] + i] : 0u;
        }
#pragma unroll
        for (int j = 0; j < kChunkSlots; j++) {
            const uint32_t i = l + 64 * j;
            if (i < chunk) stage[i] = (raw)x[j];
        }
        wave_lds_sync();
    }
#pragma unroll
    for (int k = 0; k < K; k++) {
        if (k >= kfit) break;
        store_from_stage<E>(out + (t0 + k) * kTileElems + l, g_n - (t0 + k) * kTileElems, cw[k], stage,
                            (cbase[k] - cbase[0]) + cpref[k]);
    }
    // the rest one at a time
#pragma unroll
    for (int k = 0; k < K; k++) {
        const uint64_t t = t0 + k;
        if (k < kfit) continue;
        if (t >= g_T) break;
        raw* col = out + t * kTileElems + l;
        const uint64_t rem = g_n - t * kTileElems;
        const uint64_t w = cw[k];
        const uint32_t cnt = ccnt[k];
        if (cnt <= kChunkVals) {
            wave_lds_sync();
            for (uint32_t i = l; i < cnt; i += 64) stage[i] = A[cbase[k] + i];
            wave_lds_sync();
            store_from_stage<E>(col, rem, w, stage, cpref[k]);
        } else {
            // dense tile: 16 columns at a time; their values (contiguous in A,
            // at most 1024) are staged with coalesced loads, then the group's
            // lanes write their columns
            const uint32_t myp = cpref[k];
#pragma unroll 1
            for (int h = 0; h < 4; h++) {
                const uint32_t c0 = 16u * h;
                const uint32_t lo = lane_bcast(myp, c0);
                const uint32_t hi = h == 3 ? cnt : lane_bcast(myp, c0 + 16);
                wave_lds_sync();
                stage_values<E>(A + cbase[k] + lo, hi - lo, stage);
                wave_lds_sync();
                if (l >= c0 && l < c0 + 16) store_from_stage<E>(col, rem, w, stage, myp - lo);
            }
        }
    }
}

template <class E, int K>
__device__ __forceinline__ void gather_body(const DevOperand& op, uint8_t* out_part, uint64_t n, uint64_t T,
                                            WsCtrl* ctrl) {
    using raw = typename E::raw;
    __shared__ __attribute__((aligned(16))) raw stage_all[kWavesPerBlock][kChunkVals];
    __shared__ uint32_t s_ok, s_fmt;
    __shared__ uint64_t s_nnz;
    const uint32_t wave = threadIdx.x >> 6;
    if (threadIdx.x == 0) {
        if (op.hdr) {
            HeaderView h = read_header(op.hdr, op.cap, n, E::dtype, -1);
            s_ok = h.ok; s_fmt = h.fmt; s_nnz = h.nnz;
            if (!h.ok && blockIdx.x == 0) set_status(ctrl, SPCCL_ERR_CORRUPT_STREAM);
        } else {
            s_ok = 1; s_fmt = kFmtDense; s_nnz = 0;
        }
    }
    __syncthreads();
    if (!s_ok) return;
    const uint64_t t0 = ((uint64_t)blockIdx.x * kWavesPerBlock + wave) * K;
    if (t0 >= T) return;
    raw* out = reinterpret_cast<raw*>(out_part);
    const uint8_t* d = op.hdr ? op.hdr + kHeaderBytes : op.data;
    expand_tiles<E, K>(op.data, d, s_fmt, s_nnz, n, T, t0, out, stage_all[wave], ctrl);
}

template <class E, int K>
__global__ void __launch_bounds__(kBlockThreads) k_gather(GatherArgs g) {
    gather_body<E, K>(g.part[blockIdx.y], g.out + (uint64_t)blockIdx.y * g.n * sizeof(typename E::raw), g.n, g.T,
                      g.ctrl);
}

// One all-gather hop for a batch of ranks (grid y): each rank expands its
// received message (part rebased to rb.a) into rb.out.
template <class E, int K>
__global__ void __launch_bounds__(kBlockThreads) k_gather_rb(DevOperand part, uint64_t n, WsCtrl* ctrl, RankBatch rb) {
    gather_body<E, K>(rebase(part, rb.a[blockIdx.y]), rb.out[blockIdx.y], n, num_tiles(n), ctrl);
}

// ---------------------------------------------------------------------------
// Sliced streams (Sec. III-B phase 2, Sec. V-B): every slice of kSliceElems
// elements is an independent message in its own slot.  One block of 4 waves
// owns one slice (one tile per wave): its prefix sums are block-local, so a
// single pass writes the finished message -- no look-back, no second pass --
// and the format of the slice is decided on the device from its own count.

// This wave's tile values (compacted, row order per column) to dst[0 ..
// tilecnt): through the LDS stage, in column groups when they exceed it.
template <class E>
__device__ __forceinline__ void compact_tile(const uint32_t (&v)[64], uint64_t w, uint32_t colpref,
                                             uint32_t tilecnt, typename E::raw* stage, typename E::raw* dst) {
    using raw = typename E::raw;
    const uint32_t l = lane_id();
    const bool single = tilecnt <= E::cap;
    const int ngroups = single ? 1 : E::groups;
    const uint32_t gcols = single ? 64u : E::group_cols;
#pragma unroll 1
    for (int h = 0; h < ngroups; h++) {
        const uint32_t c0 = gcols * h, c1 = c0 + gcols;
        const uint32_t lo = single ? 0u : lane_bcast(colpref, c0);
        const uint32_t hi = (single || c1 == 64) ? tilecnt : lane_bcast(colpref, c1);
        const uint64_t wm = (l >= c0 && l < c1) ? w : 0ull;
        uint32_t rank = colpref - lo;
#pragma unroll
        for (int r = 0; r < 64; r++) {
            const bool bit = (wm >> r) & 1ull;
            if (__any(bit)) {                            // rows empty in every column cost one branch
                if (bit) { stage[rank] = (raw)v[r]; rank++; }
            }
        }
        wave_lds_sync();
        for (uint32_t i = l; i < hi - lo; i += 64) dst[lo + i] = stage[i];
        wave_lds_sync();
    }
}

// out = a (+) b per slice (HasB), or a alone (compress), into a sliced
// stream (OutSliced) or a dense array.  b's slices may be Pici or dense; a
// slice of b whose header fails its check is flagged and its output slice is
// not written.
// The body works on slice q of one call's arguments, so that one launch can
// also cover the same step of several virtual ranks (k_sliced_batch).
template <class E, bool HasB, bool OutSliced>
__device__ __forceinline__ void sliced_slice(const SlicedArgs& g, uint64_t q) {
    using raw = typename E::raw;
    __shared__ raw stage_all[kWavesPerBlock][E::cap];
    __shared__ uint32_t s_cnt[kWavesPerBlock];
    const uint32_t wave = threadIdx.x >> 6, l = lane_id();
    raw* stage = stage_all[wave];
    const uint64_t base = q * kSliceElems;
    const uint64_t ns = g.n - base < kSliceElems ? g.n - base : kSliceElems;
    const uint64_t Ts = num_tiles(ns);
    const uint64_t t = wave;
    const bool has_tile = t < Ts;
    const uint8_t* a = g.a + base * sizeof(raw);
    uint32_t v[64];
    if constexpr (HasB) {
        // header and column words first (both lie inside the slot whatever
        // the header says), then half of a's rows; by then the header is in,
        // and a Pici slice's values are read early, before the other half
        // The slice's header decides the path before any other read: a
        // dense slice is a dense (+) dense pair, a Pici slice reads half of
        // a's rows, its values early (once its offsets are in), then the
        // other half.  The reads stay inside the slot (sized for a full
        // slice) or the slice's rows (a buffer resource that ends there)
        // whether or not the wave has a tile, so no branch guards them.
        const uint8_t* bm = g.b + q * g.slot;
        const HeaderView h = check_header(load_header_words(bm), g.slot, ns, E::dtype, -1);
        if (!h.ok || h.fmt == (uint32_t)kFmtCoo) {       // the same in every wave of the block
            if (threadIdx.x == 0) set_status(g.ctrl, SPCCL_ERR_CORRUPT_STREAM);
            return;
        }
        if (h.fmt != (uint32_t)kFmtPici) {
            fetch_dense<E, true>(a, t, ns, v);
            fetch_dense<E, false>(bm + kHeaderBytes, t, ns, v);
        } else {
            const PiciMeta m = load_pici_meta<E>(bm, t, ns);
            asm volatile("" ::: "memory");
            fetch_dense<E, true, 0, kEarlySplit>(a, t, ns, v);
            asm volatile("" ::: "memory");
            const EarlyVals ev = fetch_early<E>(bm, g.slot, ns, m);
            asm volatile("" ::: "memory");
            fetch_dense<E, true, kEarlySplit, 64>(a, t, ns, v);
            if (has_tile) {
                // a dense output tile that is full takes its rows as they are finished
                raw* col = (!OutSliced && ns - t * kTileElems >= kTileElems)
                               ? reinterpret_cast<raw*>(g.out) + base + t * kTileElems + l : nullptr;
                if (expand_pici_early<E, false>(pici_columns(m, h.nnz, t, ns, g.ctrl), ev, bm, ns, stage, v, col))
                    return;
            }
        }
    } else {
        if (has_tile) fetch_dense<E, true>(a, t, ns, v);
    }
    if constexpr (!OutSliced) {
        if (has_tile) store_tile<E>(g.out + base * sizeof(raw), t, ns, v);
        return;
    } else {
        const uint64_t w = has_tile ? nonzero_rows(v) : 0ull;
        const uint32_t c = (uint32_t)__popcll(w);
        const uint32_t colpref = wave_excl_scan(c);
        const uint32_t tilecnt = lane_bcast(colpref + c, 63);
        // the slice's tracker (Sec. IV-C, per slice): read by every thread
        // before the barrier, updated by one thread after it
        double s0 = 0.0, sp = 0.0;
        if (g.track && g.track_step) { s0 = g.track[2 * q]; sp = g.track[2 * q + 1]; }
        if (l == 0) s_cnt[wave] = tilecnt;
        __syncthreads();
        uint32_t tile_excl = 0, agg = 0;
#pragma unroll
        for (uint32_t k = 0; k < kWavesPerBlock; k++) {
            const uint32_t ck = s_cnt[k];
            tile_excl += k < wave ? ck : 0u;
            agg += ck;
        }
        const double meas = (double)(ns - agg) / (double)ns;
        bool dense;
        if (g.track && g.track_step) {
            const double est = sp * s0;                               // Eq. 7
            dense = est <= g.thresh;
            if (threadIdx.x == 0) g.track[2 * q + 1] = dense ? est : meas;
        } else {
            dense = meas <= g.thresh;
            if (g.track && threadIdx.x == 0) { g.track[2 * q] = meas; g.track[2 * q + 1] = meas; }
        }
        if (g.fmt_out && threadIdx.x == 0) g.fmt_out[q] = (uint8_t)(dense ? kFmtDense : kFmtPici);
        uint8_t* om = g.out + q * g.slot;
        if (dense) {                                               // this slice goes dense
            if (has_tile) store_tile<E>(om + kHeaderBytes, t, ns, v);
            if (threadIdx.x == 0)
                write_header(om, kFmtDense, E::dtype, ns, kNnzUnknown, 0, kHeaderBytes, dense_msg_bytes(ns, E::dtype));
            return;
        }
        const uint64_t oI = off_I(ns), oA = off_A(ns);
        uint32_t* I = reinterpret_cast<uint32_t*>(om + oI);
        if (has_tile) {
            reinterpret_cast<uint64_t*>(om + kHeaderBytes)[t * 64 + l] = w;
            compact_tile<E>(v, w, colpref, tilecnt, stage, reinterpret_cast<raw*>(om + oA) + tile_excl);
            if (l == 0) I[t] = tile_excl;
        }
        if (threadIdx.x == 0) {
            I[Ts] = agg;
            for (uint64_t b = oI + 4 * (Ts + 1); b < oA; b += 4) *reinterpret_cast<uint32_t*>(om + b) = 0u;
            write_header(om, kFmtPici, E::dtype, ns, agg, oI, oA, oA + (uint64_t)agg * sizeof(raw));
        }
    }
}

template <class E, bool HasB, bool OutSliced>
__global__ void __launch_bounds__(kBlockThreads) k_sliced(SlicedArgs g) {
    sliced_slice<E, HasB, OutSliced>(g, blockIdx.x);
}

// One step of the sliced ring for a batch of virtual ranks: blockIdx.y is
// the rank, whose arguments are the batch's base arguments with its own dense
// pointers, threshold and strided streams, trackers and format records.
template <class E, bool HasB, bool OutSliced>
__global__ void __launch_bounds__(kBlockThreads) k_sliced_batch(SlicedBatch b) {
    sliced_slice<E, HasB, OutSliced>(batch_rank(b, blockIdx.y), blockIdx.x);
}

// Expansion of a sliced stream: two waves per slice, each expanding two of
// its up to 4 tiles with all reads before the first store (as the gather
// does; one wave for all four was slower).  A slice whose header fails its
// check is flagged and not written.
constexpr uint32_t kExpandWavesPerSlice = 2;

template <class E>
__device__ __forceinline__ void expand_slice(const SlicedArgs& g) {
    using raw = typename E::raw;
    constexpr uint32_t K = kTilesPerPart / kExpandWavesPerSlice;
    __shared__ raw stage_all[kWavesPerBlock][kChunkVals];
    const uint32_t wave = threadIdx.x >> 6;
    const uint64_t wq = (uint64_t)blockIdx.x * kWavesPerBlock + wave;
    const uint64_t q = wq / kExpandWavesPerSlice, t0 = K * (wq % kExpandWavesPerSlice);
    if (q >= num_slices(g.n)) return;
    const uint64_t base = q * kSliceElems;
    const uint64_t ns = g.n - base < kSliceElems ? g.n - base : kSliceElems;
    if (t0 >= num_tiles(ns)) return;                      // a short last slice
    const uint8_t* bm = g.a + q * g.slot;
    const HeaderView h = check_header(load_header_words(bm), g.slot, ns, E::dtype, -1);
    if (!h.ok || h.fmt == (uint32_t)kFmtCoo) {           // slices are Pici or dense
        if (lane_id() == 0) set_status(g.ctrl, SPCCL_ERR_CORRUPT_STREAM);
        return;
    }
    expand_tiles<E, K>(bm, bm + kHeaderBytes, h.fmt, h.nnz, ns, num_tiles(ns), t0,
                       reinterpret_cast<raw*>(g.out) + base, stage_all[wave], g.ctrl);
}

template <class E>
__global__ void __launch_bounds__(kBlockThreads) k_expand_sliced(SlicedArgs g) {
    expand_slice<E>(g);
}

// One all-gather hop's expansions for a batch of virtual ranks (blockIdx.y).
template <class E>
__global__ void __launch_bounds__(kBlockThreads) k_expand_sliced_batch(SlicedBatch b) {
    expand_slice<E>(batch_rank(b, blockIdx.y));
}

// The virtual-rank send of a sliced stream: each slot's header.total_bytes,
// read on the device; one wave per slot, eight 16-byte loads per lane in
// flight before their stores, the last partial 16 bytes bytewise.  A slot whose header is not a message that
// fits is flagged and not copied.
__device__ __forceinline__ void copy_slice(const SlicedArgs& g, uint64_t nslices) {
    const uint32_t wave = threadIdx.x >> 6, l = lane_id();
    const uint64_t q = (uint64_t)blockIdx.x * kWavesPerBlock + wave;
    if (q >= nslices) return;
    const uint8_t* src = g.a + q * g.slot;
    uint8_t* dst = g.out + q * g.slot;
    const HeaderWords hw = load_header_words(src);
    const uint64_t total = hw.w[5];
    if ((uint32_t)hw.w[0] != kMagic || total < kHeaderBytes || total > g.slot) {
        if (l == 0) set_status(g.ctrl, SPCCL_ERR_CORRUPT_STREAM);
        return;
    }
    const uint4* s4 = reinterpret_cast<const uint4*>(src);
    uint4* d4 = reinterpret_cast<uint4*>(dst);
    const uint32_t nvec = (uint32_t)(total / 16);
    for (uint32_t i0 = l; i0 < nvec; i0 += 64 * 8) {
        uint4 x[8];
#pragma unroll
        for (int u = 0; u < 8; u++) x[u] = i0 + 64 * u < nvec ? s4[i0 + 64 * u] : uint4{0, 0, 0, 0};
#pragma unroll
        for (int u = 0; u < 8; u++)
            if (i0 + 64 * u < nvec) d4[i0 + 64 * u] = x[u];
    }
    const uint32_t tail = (uint32_t)(total & 15u);      // a Pici message ends on an element boundary
    if (l < tail) dst[16ull * nvec + l] = src[16ull * nvec + l];
}

__global__ void __launch_bounds__(kBlockThreads) k_copy_sliced(SlicedArgs g, uint64_t nslices) {
    copy_slice(g, nslices);
}

// The sends of one ring step for a batch of virtual ranks (blockIdx.y).
__global__ void __launch_bounds__(kBlockThreads) k_copy_sliced_batch(SlicedBatch b, uint64_t nslices) {
    copy_slice(batch_rank(b, blockIdx.y), nslices);
}

// ---------------------------------------------------------------------------
// Format decisions of the canonical ring on the device (Sec. IV-C), one
// thread per rank, between the launches of a ring step: the same rule, in
// the same IEEE double arithmetic, as the host's.  Sparsity = (m - nnz) / m;
// a send is dense iff its sparsity (first send) or the estimate sigma_prev *
// sigma0 (Eq. 7, later sends) is <= the link's threshold; a dense send tracks
// the estimate, a Pici one its measured sparsity.  Each rank's trace entry
// is written once its values are known: a Pici send's size and count by the
// next decision, when its header is in.

__device__ __forceinline__ double ring_sparsity(uint64_t m, uint64_t nnz) {
    return m == 0 ? 1.0 : (double)(m - nnz) / (double)m;
}

__device__ __forceinline__ bool ring_dense(const RingArgs& a, double sigma, double tau) {
    if (a.adaptive == 0) return false;
    if (a.adaptive == 2) return true;
    return sigma <= tau;
}

__device__ __forceinline__ double ring_tau(const RingArgs& a, int r) {
    const int rpn = a.ranks_per_node > 0 ? a.ranks_per_node : a.P;
    return ((r + 1) % rpn == 0 && rpn < a.P) ? a.inter : a.intra;
}

__device__ __forceinline__ void put_entry(spccl_trace_t* e, int step, int rank, int fmt, int measured, uint64_t bytes,
                                          uint64_t nnz, double sigma) {
    e->step = step; e->rank = rank; e->fmt = fmt; e->measured = measured;
    e->bytes = bytes; e->nnz = nnz; e->sigma = sigma;
}

__global__ void __launch_bounds__(256) k_ring_decide(RingArgs a) {
    spccl_trace_t* tr = static_cast<spccl_trace_t*>(a.trace);
    const int P = a.P;
    const uint64_t dense_bytes = dense_msg_bytes(a.m, a.dtype);
    for (int r = (int)(blockIdx.x * blockDim.x + threadIdx.x); r < P; r += (int)(gridDim.x * blockDim.x)) {
        RingRank& q = a.rr[r];
        const HeaderWords h = load_header_words(a.slots0 + (uint64_t)r * a.slot_bytes);
        const uint32_t fmt = (uint32_t)(h.w[0] >> 32) & 0xFFFFu;
        const uint64_t nnz = h.w[2], total = h.w[5];
        if (a.mode == kDecideFirst) {
            const double sg = ring_sparsity(a.m, nnz);
            const bool dense = ring_dense(a, sg, ring_tau(a, r));
            q.sigma0 = q.sigma_prev = sg;
            q.in_fmt = -1;
            q.out_fmt = dense ? kFmtDense : kFmtPici;
            put_entry(&tr[r], 0, r, q.out_fmt, 1, dense ? dense_bytes : total, nnz, sg);
        } else if (a.mode == kDecideStep) {
            const int s = a.step;
            if (s >= 2 && q.out_fmt == kFmtPici) {          // the previous send was measured
                const double sg = ring_sparsity(a.m, nnz);
                q.sigma_prev = sg;
                put_entry(&tr[(s - 1) * P + r], s - 1, r, kFmtPici, 1, total, nnz, sg);
            }
            const HeaderWords hp = load_header_words(a.slots0 + (uint64_t)((r - 1 + P) % P) * a.slot_bytes);
            q.in_fmt = (int32_t)((uint32_t)(hp.w[0] >> 32) & 0xFFFFu);   // what rank r receives now
            if (s <= P - 2) {
                const double est = q.sigma_prev * q.sigma0;
                const bool dense = ring_dense(a, est, ring_tau(a, r));
                q.out_fmt = dense ? kFmtDense : kFmtPici;
                if (dense) {
                    q.sigma_prev = est;
                    put_entry(&tr[s * P + r], s, r, kFmtDense, 0, dense_bytes, kNnzUnknown, est);
                }
            } else {
                q.out_fmt = -1;                              // the last step reduces into the output
            }
        } else if (a.mode == kDecideGather) {
            const double est = q.sigma_prev * q.sigma0;
            const bool dense = a.adaptive == 2 ? true : (a.adaptive == 0 ? false : est <= a.ag);
            q.out_fmt = dense ? kFmtDense : kFmtPici;
            put_entry(&tr[P * (P - 1) + r], P - 1, r, q.out_fmt, dense ? 0 : 1, dense_bytes, kNnzUnknown, est);
        } else if (a.mode == kDecideGatherSizes) {
            if (q.out_fmt == kFmtPici) {
                tr[P * (P - 1) + r].bytes = total;
                tr[P * (P - 1) + r].nnz = nnz;
            }
        } else {
            (void)fmt;
            put_entry(&tr[r], 0, r, kFmtPici, 1, total, nnz, ring_sparsity(a.m, nnz));
        }
    }
}

// ---------------------------------------------------------------------------
// dense (+) dense -> dense, 16 bytes per lane per step (the dense ring step)

template <class E>
__device__ __forceinline__ void dense_dense_body(const uint8_t* a_hdr, const uint8_t* a, uint64_t a_cap,
                                                 const uint8_t* b_hdr, const uint8_t* b, uint64_t b_cap,
                                                 uint8_t* out_hdr, uint8_t* out, uint64_t n, WsCtrl* ctrl) {
    using raw = typename E::raw;
    __shared__ uint32_t s_ok;
    if (threadIdx.x == 0) {
        bool ok = true;
        if (a_hdr) ok = ok && read_header(a_hdr, a_cap, n, E::dtype, kFmtDense).ok;
        if (b_hdr) ok = ok && read_header(b_hdr, b_cap, n, E::dtype, kFmtDense).ok;
        s_ok = ok;
        if (!ok && blockIdx.x == 0) set_status(ctrl, SPCCL_ERR_CORRUPT_STREAM);
        if (ok && blockIdx.x == 0 && out_hdr)
            write_header(out_hdr, kFmtDense, E::dtype, n, kNnzUnknown, 0, kHeaderBytes, dense_msg_bytes(n, E::dtype));
    }
    __syncthreads();
    if (!s_ok) return;
    constexpr uint32_t per = 16 / sizeof(raw);
    const bool vec_ok = ((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b) |
                          reinterpret_cast<uintptr_t>(out)) & 15u) == 0;
    const uint64_t nvec = vec_ok ? n / per : 0;
    const uint4* av = reinterpret_cast<const uint4*>(a);
    const uint4* bv = reinterpret_cast<const uint4*>(b);
    uint4* ov = reinterpret_cast<uint4*>(out);
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nvec; i += stride) {
        uint4 x = av[i], y = bv[i], z;
        if constexpr (sizeof(raw) == 4) {
            z.x = oplus(E{}, x.x, y.x); z.y = oplus(E{}, x.y, y.y);
            z.z = oplus(E{}, x.z, y.z); z.w = oplus(E{}, x.w, y.w);
        } else {
            auto two = [](uint32_t p, uint32_t q) {
                return oplus(E{}, p & 0xFFFFu, q & 0xFFFFu) | (oplus(E{}, p >> 16, q >> 16) << 16);
            };
            z.x = two(x.x, y.x); z.y = two(x.y, y.y); z.z = two(x.z, y.z); z.w = two(x.w, y.w);
        }
        st_stream(&ov[i], z);
    }
    // the tail (or everything, for arrays that are not 16-byte aligned)
    const raw* ae = reinterpret_cast<const raw*>(a);
    const raw* be = reinterpret_cast<const raw*>(b);
    raw* oe = reinterpret_cast<raw*>(out);
    for (uint64_t i = nvec * per + (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        st_stream(&oe[i], (raw)oplus(E{}, ae[i], be[i]));
}

template <class E>
__global__ void __launch_bounds__(256) k_dense_dense(const uint8_t* a_hdr, const uint8_t* a, uint64_t a_cap,
                                                     const uint8_t* b_hdr, const uint8_t* b, uint64_t b_cap,
                                                     uint8_t* out_hdr, uint8_t* out, uint64_t n, WsCtrl* ctrl) {
    dense_dense_body<E>(a_hdr, a, a_cap, b_hdr, b, b_cap, out_hdr, out, n, ctrl);
}

template <class E>
__global__ void __launch_bounds__(256) k_dense_dense_rb(DenseSinkArgs g, RankBatch rb) {
    if (rank_skipped(rb, blockIdx.y)) return;
    const DenseSinkArgs r = rank_dense(g, rb, blockIdx.y);
    dense_dense_body<E>(r.a.hdr, r.a.data, r.a.cap, r.b.hdr, r.b.data, r.b.cap, r.out_hdr, r.out, g.n, g.ctrl);
}

// ---------------------------------------------------------------------------
// message copy sized on the device (the virtual-rank send)

__device__ __forceinline__ void copy_message_body(const uint8_t* src, uint64_t src_cap, uint8_t* dst,
                                                  uint64_t dst_cap, WsCtrl* ctrl) {
    __shared__ uint64_t s_total;
    if (threadIdx.x == 0) {
        uint64_t total = 0;
        if (src_cap >= kHeaderBytes) {
            const uint64_t* w = reinterpret_cast<const uint64_t*>(src);
            total = ((uint32_t)w[0] == kMagic) ? w[5] : 0;
        }
        if (total < kHeaderBytes || total > src_cap || total > dst_cap) {
            if (blockIdx.x == 0) set_status(ctrl, SPCCL_ERR_CORRUPT_STREAM);
            total = 0;
        }
        s_total = total;
    }
    __syncthreads();
    const uint64_t total = s_total;
    const uint64_t nvec = total / 16;
    const uint4* s4 = reinterpret_cast<const uint4*>(src);
    uint4* d4 = reinterpret_cast<uint4*>(dst);
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nvec; i += stride) st_stream(&d4[i], s4[i]);
    if (blockIdx.x == 0)
        for (uint64_t b = nvec * 16 + threadIdx.x; b < total; b += blockDim.x) dst[b] = src[b];
}

__global__ void __launch_bounds__(256) k_copy_message(const uint8_t* src, uint64_t src_cap, uint8_t* dst,
                                                      uint64_t dst_cap, WsCtrl* ctrl) {
    copy_message_body(src, src_cap, dst, dst_cap, ctrl);
}

// The sends of one ring step for a batch of ranks (grid y): rb.a -> rb.out.
__global__ void __launch_bounds__(256) k_copy_message_rb(uint64_t src_cap, uint64_t dst_cap, WsCtrl* ctrl,
                                                         RankBatch rb) {
    copy_message_body(rb.a[blockIdx.y], src_cap, rb.out[blockIdx.y], dst_cap, ctrl);
}

template <class E>
__device__ __forceinline__ void encode_dense_body(const uint8_t* src, uint8_t* out, uint64_t n) {
    if (blockIdx.x == 0 && threadIdx.x == 0)
        write_header(out, kFmtDense, E::dtype, n, kNnzUnknown, 0, kHeaderBytes, dense_msg_bytes(n, E::dtype));
    using raw = typename E::raw;
    const uint64_t bytes = n * sizeof(raw);
    const bool vec_ok = (reinterpret_cast<uintptr_t>(src) & 15u) == 0;
    const uint64_t nvec = vec_ok ? bytes / 16 : 0;
    const uint4* s4 = reinterpret_cast<const uint4*>(src);
    uint4* d4 = reinterpret_cast<uint4*>(out + kHeaderBytes);
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nvec; i += stride) st_stream(&d4[i], s4[i]);
    // the tail (or everything, for a source that is not 16-byte aligned), element by element
    const raw* se = reinterpret_cast<const raw*>(src);
    raw* de = reinterpret_cast<raw*>(out + kHeaderBytes);
    for (uint64_t i = nvec * 16 / sizeof(raw) + (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        st_stream(&de[i], se[i]);
}

template <class E>
__global__ void __launch_bounds__(256) k_encode_dense(const uint8_t* src, uint8_t* out, uint64_t n) {
    encode_dense_body<E>(src, out, n);
}

// Dense sends of one ring step for a batch of ranks (grid y): rb.a -> rb.out.
template <class E>
__global__ void __launch_bounds__(256) k_encode_dense_rb(uint64_t n, RankBatch rb) {
    if (rank_skipped(rb, blockIdx.y)) return;
    encode_dense_body<E>(rb.a[blockIdx.y], rb.out[blockIdx.y], n);
}

__global__ void __launch_bounds__(256) k_fill_zero(uint4* p, uint64_t nvec, uint8_t* tail, uint64_t ntail) {
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nvec; i += stride) st_stream(&p[i], uint4{0, 0, 0, 0});
    if (blockIdx.x == 0)
        for (uint64_t b = threadIdx.x; b < ntail; b += blockDim.x) tail[b] = 0;
}

// ---------------------------------------------------------------------------
// host launchers

namespace {

inline spccl_status_t launch_status() {
    return hipGetLastError() == hipSuccess ? SPCCL_OK : SPCCL_ERR_HIP;
}

inline uint32_t stream_grid(uint64_t work_items, uint32_t per_block, uint32_t cap) {
    uint64_t g = (work_items + per_block - 1) / per_block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (uint32_t)g;
}

// Which kernels write a Pici output, by its size in partitions of 16384
// elements (fp32 times at 2^k elements, isolated medians after a 512 MiB
// write, sigma 0.99 / 0.9; "one" = one launch finding its offsets by the
// two-level look-back, "two" = count pass + k_place):
//  - dense sources (k_to_pici): one launch at every size in fp32 (2^25:
//    compression 31.9 / 33.8 against 35.1 / 42.3 us, dense (+) Pici 34.9 /
//    44.0 against 38.3 / 54.9; 2^26: 57.7 / 60.7 against 58.5 / 77.3 and
//    61.1 / 78.6 against 66.7 / 98.1; 2^27: 107 / 113 against 110 / 147);
//    in bf16 up to 2048 partitions (2^25 elements: 21.4 / 23.4 against 23.1 /
//    29.1), since from 4096 the one launch loses at 0.99 (2^27: 68.2 against
//    59.1 us; at 0.9 it still wins, 74.5 against 76.4).
//  - Pici (+) Pici: one launch of the per-tile kernel up to 1024 partitions
//    (2^24: 14.8 / 29.2 against 15.5 / 31.7 us), then its two-pass form
//    (k_pp_tile<E, true> + k_place, four waves per partition: 12.7 against
//    20.1 us at 2^20 and 0.99 against one partition per wave), from 2048
//    partitions one partition per wave (k_pp_part: 28.2 against 36.3 us at
//    2^26), which finds its own offsets (with its count published before its
//    merges: 21.1 / 65.6 us at 2^26 against 28.2 / 75.2 with k_place; 38.0 /
//    126.6 against 40.9 / 144.5 at 2^27, 8192 partitions, two rounds of
//    waves).
// Without value slots (a minimal workspace) every output takes one launch.
constexpr uint32_t kOneLaunchMaxPartsBF16 = 2048;
constexpr uint32_t kPPTileOneMaxParts = 1024;
constexpr uint32_t kPPTileMaxParts = 2048;

}  // namespace

// An upper bound on the sizes above (in partitions) for calls whose
// workspace has the value slots; set by spccl_set_single_pass_limit.  0
// keeps every such call on two passes.
std::atomic<uint32_t> g_single_pass_max_parts{0xFFFFFFFFu};

uint32_t set_single_pass_max_parts(uint32_t parts) { return g_single_pass_max_parts.exchange(parts); }

namespace {

template <class E>
spccl_status_t launch_to_pici(int sa, int sb, const PiciSinkArgs& g, hipStream_t st) {
    dim3 grid(g.nparts), block(kBlockThreads);
    const uint32_t bound = g_single_pass_max_parts.load(std::memory_order_relaxed);
    const auto one_launch = [&](uint32_t max_parts) {
        return !g.slots || g.nparts <= (max_parts < bound ? max_parts : bound);
    };
    const bool two_pass = !one_launch(sizeof(typename E::raw) == 4 ? 0xFFFFFFFFu : kOneLaunchMaxPartsBF16);
    if (sa == SRC_PICI && sb == SRC_PICI) {
        if (!one_launch(kPPTileOneMaxParts)) {
            if (g.nparts < kPPTileMaxParts) {
                hipLaunchKernelGGL((k_pp_tile<E, true>), grid, block, 0, st, g);
            } else {
                dim3 wgrid((g.nparts + kWavesPerBlock - 1) / kWavesPerBlock);
                if (one_launch(0xFFFFFFFFu)) {
                    hipLaunchKernelGGL((k_pp_part<E, true>), wgrid, block, 0, st, g);
                    return launch_status();
                }
                hipLaunchKernelGGL((k_pp_part<E, false>), wgrid, block, 0, st, g);
            }
            spccl_status_t st1 = launch_status();
            if (st1 != SPCCL_OK) return st1;
            dim3 pgrid((g.nparts + kPlacePer - 1) / kPlacePer);
            hipLaunchKernelGGL(k_place<E>, pgrid, block, 0, st, g);
        } else {
            hipLaunchKernelGGL((k_pp_tile<E, false>), grid, block, 0, st, g);
        }
        return launch_status();
    }
    if (two_pass) {
#define SPCCL_TO_PICI2(A, B) hipLaunchKernelGGL((k_to_pici<E, A, B, true>), grid, block, 0, st, g)
        if (sa == SRC_DENSE && sb == SRC_NONE) SPCCL_TO_PICI2(SRC_DENSE, SRC_NONE);
        else if (sa == SRC_DENSE && sb == SRC_DENSE) SPCCL_TO_PICI2(SRC_DENSE, SRC_DENSE);
        else if (sa == SRC_DENSE && sb == SRC_PICI) SPCCL_TO_PICI2(SRC_DENSE, SRC_PICI);
        else if (sa == SRC_PICI && sb == SRC_DENSE) SPCCL_TO_PICI2(SRC_PICI, SRC_DENSE);
        else return SPCCL_ERR_UNSUPPORTED;
#undef SPCCL_TO_PICI2
        spccl_status_t st1 = launch_status();
        if (st1 != SPCCL_OK) return st1;
        dim3 pgrid((g.nparts + kPlacePer - 1) / kPlacePer);
        hipLaunchKernelGGL(k_place<E>, pgrid, block, 0, st, g);
        return launch_status();
    }
#define SPCCL_TO_PICI(A, B) hipLaunchKernelGGL((k_to_pici<E, A, B, false>), grid, block, 0, st, g)
    if (sa == SRC_DENSE && sb == SRC_NONE) SPCCL_TO_PICI(SRC_DENSE, SRC_NONE);
    else if (sa == SRC_DENSE && sb == SRC_DENSE) SPCCL_TO_PICI(SRC_DENSE, SRC_DENSE);
    else if (sa == SRC_DENSE && sb == SRC_PICI) SPCCL_TO_PICI(SRC_DENSE, SRC_PICI);
    else if (sa == SRC_PICI && sb == SRC_DENSE) SPCCL_TO_PICI(SRC_PICI, SRC_DENSE);
    else return SPCCL_ERR_UNSUPPORTED;
#undef SPCCL_TO_PICI
    return launch_status();
}

// COO sink: count pass, then the place pass (offsets and total from chunk sums).
template <class E>
spccl_status_t launch_to_coo(int sa, int sb, const PiciSinkArgs& g, hipStream_t st) {
    dim3 grid(g.nparts), block(kBlockThreads);
#define SPCCL_TO_COO(A, B) hipLaunchKernelGGL((k_to_coo<E, A, B>), grid, block, 0, st, g)
    if (sa == SRC_DENSE && sb == SRC_NONE) SPCCL_TO_COO(SRC_DENSE, SRC_NONE);
    else if (sa == SRC_DENSE && sb == SRC_DENSE) SPCCL_TO_COO(SRC_DENSE, SRC_DENSE);
    else if (sa == SRC_DENSE && sb == SRC_COO) SPCCL_TO_COO(SRC_DENSE, SRC_COO);
    else if (sa == SRC_COO && sb == SRC_DENSE) SPCCL_TO_COO(SRC_COO, SRC_DENSE);
    else if (sa == SRC_COO && sb == SRC_COO) SPCCL_TO_COO(SRC_COO, SRC_COO);
    else return SPCCL_ERR_UNSUPPORTED;
#undef SPCCL_TO_COO
    spccl_status_t st1 = launch_status();
    if (st1 != SPCCL_OK) return st1;
    hipLaunchKernelGGL(k_place_coo<E>, dim3((g.nparts + kWavesPerBlock - 1) / kWavesPerBlock), block, 0, st, g);
    return launch_status();
}

template <class E>
spccl_status_t launch_to_dense(int sa, int sb, const DenseSinkArgs& g, hipStream_t st) {
    dim3 grid(stream_grid(g.T, kWavesPerBlock, 0x7FFFFFFF)), block(kBlockThreads);
#define SPCCL_TO_DENSE(A, B) hipLaunchKernelGGL((k_to_dense<E, A, B>), grid, block, 0, st, g)
    if (sa == SRC_DENSE && sb == SRC_PICI) SPCCL_TO_DENSE(SRC_DENSE, SRC_PICI);
    else if (sa == SRC_PICI && sb == SRC_DENSE) SPCCL_TO_DENSE(SRC_PICI, SRC_DENSE);
    else if (sa == SRC_PICI && sb == SRC_PICI) SPCCL_TO_DENSE(SRC_PICI, SRC_PICI);
    else if (sa == SRC_PICI && sb == SRC_NONE) SPCCL_TO_DENSE(SRC_PICI, SRC_NONE);
    else if (sa == SRC_DENSE && sb == SRC_COO) SPCCL_TO_DENSE(SRC_DENSE, SRC_COO);
    else if (sa == SRC_COO && sb == SRC_DENSE) SPCCL_TO_DENSE(SRC_COO, SRC_DENSE);
    else if (sa == SRC_COO && sb == SRC_COO) SPCCL_TO_DENSE(SRC_COO, SRC_COO);
    else if (sa == SRC_COO && sb == SRC_NONE) SPCCL_TO_DENSE(SRC_COO, SRC_NONE);
    else return SPCCL_ERR_UNSUPPORTED;
#undef SPCCL_TO_DENSE
    return launch_status();
}

}  // namespace

spccl_status_t launch_to_pici_dt(int dtype, int sa, int sb, const PiciSinkArgs& g, hipStream_t st) {
    return dtype == kBF16 ? launch_to_pici<BF16>(sa, sb, g, st) : launch_to_pici<F32>(sa, sb, g, st);
}

spccl_status_t launch_to_dense_dt(int dtype, int sa, int sb, const DenseSinkArgs& g, hipStream_t st) {
    return dtype == kBF16 ? launch_to_dense<BF16>(sa, sb, g, st) : launch_to_dense<F32>(sa, sb, g, st);
}

spccl_status_t launch_to_coo_dt(int dtype, int sa, int sb, const PiciSinkArgs& g, hipStream_t st) {
    return dtype == kBF16 ? launch_to_coo<BF16>(sa, sb, g, st) : launch_to_coo<F32>(sa, sb, g, st);
}

// Tiles per wave of the expansion: two once that still leaves enough waves
// to fill the chip (about 8192 resident), else one.  Four tiles per wave
// measured the same at 99% sparsity and 10% slower at 90% (their values no
// longer fit one staged chunk), one tile per wave 5-10% slower at 99%.
template <class E>
void launch_gather_k(const GatherArgs& g, int P, hipStream_t st) {
    const uint64_t tiles = g.T * (uint64_t)P;
    const int K = tiles >= 2 * 8192 ? 2 : 1;
    dim3 block(kBlockThreads);
    dim3 grid(stream_grid(g.T, kWavesPerBlock * K, 0x7FFFFFFF), (unsigned)P);
    if (K == 2) hipLaunchKernelGGL((k_gather<E, 2>), grid, block, 0, st, g);
    else hipLaunchKernelGGL((k_gather<E, 1>), grid, block, 0, st, g);
}

spccl_status_t launch_gather_dt(int dtype, const GatherArgs& g, int P, hipStream_t st) {
    if (dtype == kBF16) launch_gather_k<BF16>(g, P, st);
    else launch_gather_k<F32>(g, P, st);
    return launch_status();
}

spccl_status_t launch_dense_dense_dt(int dtype, const uint8_t* a_hdr, const uint8_t* a, uint64_t a_cap,
                                     const uint8_t* b_hdr, const uint8_t* b, uint64_t b_cap, uint8_t* out_hdr,
                                     uint8_t* out, uint64_t n, WsCtrl* ctrl, hipStream_t st) {
    const uint64_t vec = n / (16 / elem_bytes(dtype));
    dim3 grid(stream_grid(vec, 256 * 4, 8192)), block(256);
    if (dtype == kBF16)
        hipLaunchKernelGGL(k_dense_dense<BF16>, grid, block, 0, st, a_hdr, a, a_cap, b_hdr, b, b_cap, out_hdr, out, n, ctrl);
    else
        hipLaunchKernelGGL(k_dense_dense<F32>, grid, block, 0, st, a_hdr, a, a_cap, b_hdr, b, b_cap, out_hdr, out, n, ctrl);
    return launch_status();
}

spccl_status_t launch_copy_message(const uint8_t* src, uint64_t src_cap, uint8_t* dst, uint64_t dst_cap,
                                   WsCtrl* ctrl, hipStream_t st) {
    const uint64_t cap = src_cap < dst_cap ? src_cap : dst_cap;
    dim3 grid(stream_grid(cap / 16, 256 * 4, 4096)), block(256);
    hipLaunchKernelGGL(k_copy_message, grid, block, 0, st, src, src_cap, dst, dst_cap, ctrl);
    return launch_status();
}

spccl_status_t launch_encode_dense_dt(int dtype, const uint8_t* src, uint8_t* out, uint64_t n, hipStream_t st) {
    dim3 grid(stream_grid(n * elem_bytes(dtype) / 16, 256 * 4, 4096)), block(256);
    if (dtype == kBF16) hipLaunchKernelGGL(k_encode_dense<BF16>, grid, block, 0, st, src, out, n);
    else hipLaunchKernelGGL(k_encode_dense<F32>, grid, block, 0, st, src, out, n);
    return launch_status();
}

template <class E>
void launch_sliced_t(const SlicedArgs& g, int op, hipStream_t st) {
    const uint64_t S = num_slices(g.n);
    dim3 block(kBlockThreads);
    if (op == kSlicedCompress) hipLaunchKernelGGL((k_sliced<E, false, true>), dim3(S), block, 0, st, g);
    else if (op == kSlicedReduceToSliced) hipLaunchKernelGGL((k_sliced<E, true, true>), dim3(S), block, 0, st, g);
    else if (op == kSlicedReduceToDense) hipLaunchKernelGGL((k_sliced<E, true, false>), dim3(S), block, 0, st, g);
    else hipLaunchKernelGGL(k_expand_sliced<E>,
                            dim3((S * kExpandWavesPerSlice + kWavesPerBlock - 1) / kWavesPerBlock), block, 0, st, g);
}

spccl_status_t launch_sliced_dt(int dtype, const SlicedArgs& g, int op, hipStream_t st) {
    if (dtype == kBF16) launch_sliced_t<BF16>(g, op, st);
    else launch_sliced_t<F32>(g, op, st);
    return launch_status();
}

template <class E>
void launch_sliced_batch_t(const SlicedBatch& b, uint32_t ranks, int op, hipStream_t st) {
    const uint64_t S = num_slices(b.base.n);
    const dim3 grid((unsigned)S, ranks), block(kBlockThreads);
    if (op == kSlicedExpand)
        hipLaunchKernelGGL(k_expand_sliced_batch<E>,
                           dim3((unsigned)((S * kExpandWavesPerSlice + kWavesPerBlock - 1) / kWavesPerBlock), ranks),
                           block, 0, st, b);
    else if (op == kSlicedCompress) hipLaunchKernelGGL((k_sliced_batch<E, false, true>), grid, block, 0, st, b);
    else if (op == kSlicedReduceToSliced) hipLaunchKernelGGL((k_sliced_batch<E, true, true>), grid, block, 0, st, b);
    else hipLaunchKernelGGL((k_sliced_batch<E, true, false>), grid, block, 0, st, b);
}

spccl_status_t launch_sliced_batch_dt(int dtype, const SlicedBatch& b, uint32_t ranks, int op, hipStream_t st) {
    if (ranks == 0 || ranks > (uint32_t)kMaxBatchRanks) return SPCCL_ERR_INVALID_ARG;
    if (dtype == kBF16) launch_sliced_batch_t<BF16>(b, ranks, op, st);
    else launch_sliced_batch_t<F32>(b, ranks, op, st);
    return launch_status();
}

spccl_status_t launch_copy_sliced_batch(const SlicedBatch& b, uint32_t ranks, hipStream_t st) {
    if (ranks == 0 || ranks > (uint32_t)kMaxBatchRanks) return SPCCL_ERR_INVALID_ARG;
    const uint64_t S = num_slices(b.base.n);
    hipLaunchKernelGGL(k_copy_sliced_batch, dim3((unsigned)((S + kWavesPerBlock - 1) / kWavesPerBlock), ranks),
                       dim3(kBlockThreads), 0, st, b, S);
    return launch_status();
}

// ---- batched launches of one canonical ring step (grid y = rank) ----------
// Grid-stride kernels give each rank a share of about 4096 blocks.
inline uint32_t per_rank_cap(uint32_t ranks) { return ranks >= 64 ? 64u : 4096u / ranks; }

template <class E, bool Deferred>
spccl_status_t launch_to_pici_rb_k(int sa, int sb, const PiciSinkArgs& g, const RankBatch& rb, uint32_t ranks,
                                   hipStream_t st) {
    const dim3 grid(g.nparts, ranks), block(kBlockThreads);
#define SPCCL_TO_PICI_RB(A, B) hipLaunchKernelGGL((k_to_pici_rb<E, A, B, Deferred>), grid, block, 0, st, g, rb)
    if (sa == SRC_DENSE && sb == SRC_NONE) SPCCL_TO_PICI_RB(SRC_DENSE, SRC_NONE);
    else if (sa == SRC_PICI && sb == SRC_DENSE) SPCCL_TO_PICI_RB(SRC_PICI, SRC_DENSE);
    else if (sa == SRC_DENSE && sb == SRC_DENSE) SPCCL_TO_PICI_RB(SRC_DENSE, SRC_DENSE);
    else return SPCCL_ERR_UNSUPPORTED;
#undef SPCCL_TO_PICI_RB
    return launch_status();
}

// The same choice as launch_to_pici, per rank's message.
template <class E>
spccl_status_t launch_to_pici_rb(int sa, int sb, const PiciSinkArgs& g, const RankBatch& rb, uint32_t ranks,
                                 hipStream_t st) {
    const uint32_t bound = g_single_pass_max_parts.load(std::memory_order_relaxed);
    const uint32_t own = sizeof(typename E::raw) == 4 ? 0xFFFFFFFFu : kOneLaunchMaxPartsBF16;
    if (g.nparts <= (own < bound ? own : bound)) return launch_to_pici_rb_k<E, false>(sa, sb, g, rb, ranks, st);
    spccl_status_t s1 = launch_to_pici_rb_k<E, true>(sa, sb, g, rb, ranks, st);
    if (s1 != SPCCL_OK) return s1;
    hipLaunchKernelGGL(k_place_rb<E>, dim3((g.nparts + kPlacePer - 1) / kPlacePer, ranks), dim3(kBlockThreads), 0, st,
                       g, rb);
    return launch_status();
}

template <class E>
spccl_status_t launch_to_dense_rb(int sa, int sb, const DenseSinkArgs& g, const RankBatch& rb, uint32_t ranks,
                                  hipStream_t st) {
    if (sa == SRC_DENSE && sb == SRC_DENSE) {
        const uint64_t vec = g.n / (16 / sizeof(typename E::raw));
        hipLaunchKernelGGL(k_dense_dense_rb<E>, dim3(stream_grid(vec, 256 * 4, per_rank_cap(ranks)), ranks), dim3(256), 0,
                           st, g, rb);
    } else if (sa == SRC_PICI && sb == SRC_DENSE) {
        hipLaunchKernelGGL((k_to_dense_rb<E, SRC_PICI, SRC_DENSE>),
                           dim3(stream_grid(g.T, kWavesPerBlock, 0x7FFFFFFF), ranks), dim3(kBlockThreads), 0, st, g, rb);
    } else {
        return SPCCL_ERR_UNSUPPORTED;
    }
    return launch_status();
}

spccl_status_t launch_to_pici_rb_dt(int dtype, int sa, int sb, const PiciSinkArgs& g, const RankBatch& rb,
                                    uint32_t ranks, hipStream_t st) {
    if (ranks == 0 || ranks > (uint32_t)kMaxBatchRanks || !g.slots) return SPCCL_ERR_INVALID_ARG;
    return dtype == kBF16 ? launch_to_pici_rb<BF16>(sa, sb, g, rb, ranks, st)
                          : launch_to_pici_rb<F32>(sa, sb, g, rb, ranks, st);
}

spccl_status_t launch_to_dense_rb_dt(int dtype, int sa, int sb, const DenseSinkArgs& g, const RankBatch& rb,
                                     uint32_t ranks, hipStream_t st) {
    if (ranks == 0 || ranks > (uint32_t)kMaxBatchRanks) return SPCCL_ERR_INVALID_ARG;
    return dtype == kBF16 ? launch_to_dense_rb<BF16>(sa, sb, g, rb, ranks, st)
                          : launch_to_dense_rb<F32>(sa, sb, g, rb, ranks, st);
}

spccl_status_t launch_copy_message_rb(uint64_t src_cap, uint64_t dst_cap, WsCtrl* ctrl, const RankBatch& rb,
                                      uint32_t ranks, hipStream_t st) {
    if (ranks == 0 || ranks > (uint32_t)kMaxBatchRanks) return SPCCL_ERR_INVALID_ARG;
    const uint64_t cap = src_cap < dst_cap ? src_cap : dst_cap;
    hipLaunchKernelGGL(k_copy_message_rb, dim3(stream_grid(cap / 16, 256 * 4, per_rank_cap(ranks)), ranks), dim3(256),
                       0, st, src_cap, dst_cap, ctrl, rb);
    return launch_status();
}

spccl_status_t launch_encode_dense_rb_dt(int dtype, uint64_t n, const RankBatch& rb, uint32_t ranks, hipStream_t st) {
    if (ranks == 0 || ranks > (uint32_t)kMaxBatchRanks) return SPCCL_ERR_INVALID_ARG;
    const dim3 grid(stream_grid(n * elem_bytes(dtype) / 16, 256 * 4, per_rank_cap(ranks)), ranks), block(256);
    if (dtype == kBF16) hipLaunchKernelGGL(k_encode_dense_rb<BF16>, grid, block, 0, st, n, rb);
    else hipLaunchKernelGGL(k_encode_dense_rb<F32>, grid, block, 0, st, n, rb);
    return launch_status();
}

// One expansion per rank: rb.a[r] (a message, any format, or an array) into
// rb.out[r]; part gives the operand's kind (hdr null: an array) and capacity.
spccl_status_t launch_gather_rb_dt(int dtype, const DevOperand& part, uint64_t n, WsCtrl* ctrl, const RankBatch& rb,
                                   uint32_t ranks, hipStream_t st) {
    if (ranks == 0 || ranks > (uint32_t)kMaxBatchRanks) return SPCCL_ERR_INVALID_ARG;
    const uint64_t T = num_tiles(n);
    const int K = T * ranks >= 2 * 8192 ? 2 : 1;
    const dim3 grid(stream_grid(T, kWavesPerBlock * K, 0x7FFFFFFF), ranks), block(kBlockThreads);
    if (dtype == kBF16) {
        if (K == 2) hipLaunchKernelGGL((k_gather_rb<BF16, 2>), grid, block, 0, st, part, n, ctrl, rb);
        else hipLaunchKernelGGL((k_gather_rb<BF16, 1>), grid, block, 0, st, part, n, ctrl, rb);
    } else {
        if (K == 2) hipLaunchKernelGGL((k_gather_rb<F32, 2>), grid, block, 0, st, part, n, ctrl, rb);
        else hipLaunchKernelGGL((k_gather_rb<F32, 1>), grid, block, 0, st, part, n, ctrl, rb);
    }
    return launch_status();
}

spccl_status_t launch_ring_decide(const RingArgs& a, hipStream_t st) {
    hipLaunchKernelGGL(k_ring_decide, dim3((a.P + 255) / 256), dim3(256), 0, st, a);
    return launch_status();
}

// nnz <= n, and the kernel strides over the grid
spccl_status_t launch_coo_index(const uint8_t* msg, uint64_t cap, uint64_t n, int dtype, uint64_t* idx,
                                uint32_t epoch, WsCtrl* ctrl, hipStream_t st) {
    const dim3 grid(stream_grid(n + 1, 256, 4096)), block(256);
    hipLaunchKernelGGL(k_coo_index, grid, block, 0, st, msg, cap, n, dtype, idx, epoch, ctrl);
    return launch_status();
}

spccl_status_t launch_copy_sliced(const SlicedArgs& g, hipStream_t st) {
    const uint64_t S = num_slices(g.n);
    hipLaunchKernelGGL(k_copy_sliced, dim3((S + kWavesPerBlock - 1) / kWavesPerBlock), dim3(kBlockThreads), 0, st,
                       g, S);
    return launch_status();
}

spccl_status_t launch_fill_zero(void* p, uint64_t bytes, hipStream_t st) {
    const uint64_t nvec = bytes / 16;
    dim3 grid(stream_grid(nvec, 256 * 4, 4096)), block(256);
    hipLaunchKernelGGL(k_fill_zero, grid, block, 0, st, reinterpret_cast<uint4*>(p), nvec,
                       reinterpret_cast<uint8_t*>(p) + nvec * 16, bytes - nvec * 16);
    return launch_status();
}

}  // namespace spccl
