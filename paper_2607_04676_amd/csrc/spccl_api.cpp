// C ABI entry points: host-side argument checks, operand decoding and kernel
// dispatch.  Nothing here allocates device memory or synchronizes, except
// spccl_read_header / spccl_read_status.
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <string.h>

#include <atomic>

#include "spccl_internal.h"
#include "../../include/spccl.h"

namespace spccl {
spccl_status_t launch_to_pici_dt(int dtype, int sa, int sb, const PiciSinkArgs& g, hipStream_t st);
spccl_status_t launch_to_dense_dt(int dtype, int sa, int sb, const DenseSinkArgs& g, hipStream_t st);
spccl_status_t launch_to_coo_dt(int dtype, int sa, int sb, const PiciSinkArgs& g, hipStream_t st);
spccl_status_t launch_gather_dt(int dtype, const GatherArgs& g, int P, hipStream_t st);
spccl_status_t launch_dense_dense_dt(int dtype, const uint8_t* a_hdr, const uint8_t* a, uint64_t a_cap,
                                     const uint8_t* b_hdr, const uint8_t* b, uint64_t b_cap, uint8_t* out_hdr,
                                     uint8_t* out, uint64_t n, WsCtrl* ctrl, hipStream_t st);
spccl_status_t launch_copy_message(const uint8_t* src, uint64_t src_cap, uint8_t* dst, uint64_t dst_cap,
                                   WsCtrl* ctrl, hipStream_t st);
spccl_status_t launch_fill_zero(void* p, uint64_t bytes, hipStream_t st);
spccl_status_t launch_encode_dense_dt(int dtype, const uint8_t* src, uint8_t* out, uint64_t n, hipStream_t st);
spccl_status_t launch_sliced_dt(int dtype, const SlicedArgs& g, int op, hipStream_t st);
spccl_status_t launch_copy_sliced(const SlicedArgs& g, hipStream_t st);
spccl_status_t launch_coo_index(const uint8_t* msg, uint64_t cap, uint64_t n, int dtype, uint64_t* idx,
                                uint32_t epoch, WsCtrl* ctrl, hipStream_t st);
uint32_t set_single_pass_max_parts(uint32_t parts);
}  // namespace spccl

namespace spccl {
// Every launch that publishes look-back words tags them with a fresh epoch,
// so a workspace never needs clearing between calls: words left by earlier
// calls carry other epochs (30 bits; a word would have to go unwritten for
// 2^30 launches to be mistaken).
static std::atomic<uint32_t> g_epoch{1};
uint32_t next_epoch() { return g_epoch.fetch_add(1, std::memory_order_relaxed) & 0x3FFFFFFFu; }
}  // namespace spccl

using namespace spccl;

namespace {

inline bool dtype_ok(int32_t dt) { return dt == kF32 || dt == kBF16; }
inline uint64_t align256(uint64_t x) { return (x + 255ull) & ~255ull; }
// Workspace regions: control block, look-back words, the tile indexes of two
// COO operands, value slots (the two-pass Pici sink and the COO sink), index
// slots (the COO sink).
inline uint64_t coo_index_offset(uint64_t n, int which) {
    return align256(kWsFlagsOffset + 8ull * flag_words(n)) + (uint64_t)which * align256(8ull * (num_tiles(n) + 1));
}
inline uint64_t slots_offset(uint64_t n) { return coo_index_offset(n, 2); }
inline uint64_t value_slots_end(uint64_t n, int32_t dt) {
    return slots_offset(n) + num_parts(n) * kPartElems * elem_bytes(dt);
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
// dense arrays need only element alignment (chunks of a rank's buffer start anywhere)
inline bool aligned_elem(const void* p, int32_t dt) {
    return (reinterpret_cast<uintptr_t>(p) & (elem_bytes(dt) - 1)) == 0;
}
inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }
inline bool overlaps(const void* a, uint64_t an, const void* b, uint64_t bn) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return an && bn && x < y + bn && y < x + an;
}

spccl_status_t check_ws(void* ws, uint64_t ws_bytes, uint64_t need) {
    if (!ws || !aligned16(ws)) return SPCCL_ERR_INVALID_ARG;
    if (ws_bytes < need) return SPCCL_ERR_WORKSPACE;
    return SPCCL_OK;
}

// An input operand as a kernel source.
struct Src {
    int kind;          // SRC_DENSE or SRC_PICI
    DevOperand dev;
};

spccl_status_t decode_input(const spccl_operand_t& o, uint64_t n, int32_t dt, Src* out) {
    if (!o.ptr) return SPCCL_ERR_INVALID_ARG;
    if (o.kind == SPCCL_ARRAY ? !aligned_elem(o.ptr, dt) : !aligned16(o.ptr)) return SPCCL_ERR_INVALID_ARG;
    const uint8_t* p = static_cast<const uint8_t*>(o.ptr);
    if (o.kind == SPCCL_ARRAY) {
        if (o.bytes < n * elem_bytes(dt)) return SPCCL_ERR_CAPACITY;
        *out = Src{SRC_DENSE, DevOperand{nullptr, p, o.bytes}};
        return SPCCL_OK;
    }
    if (o.kind != SPCCL_STREAM) return SPCCL_ERR_INVALID_ARG;
    // the smallest valid message of the declared format: kernels read a dense
    // message's values, or a Pici message's index arrays, before its header
    // has been checked
    if (o.fmt == SPCCL_FMT_DENSE) {
        if (o.bytes < dense_msg_bytes(n, dt)) return SPCCL_ERR_CAPACITY;
        *out = Src{SRC_DENSE, DevOperand{p, p + kHeaderBytes, o.bytes}};
    } else if (o.fmt == SPCCL_FMT_PICI) {
        if (o.bytes < off_A(n)) return SPCCL_ERR_CAPACITY;
        *out = Src{SRC_PICI, DevOperand{p, p, o.bytes}};
    } else if (o.fmt == SPCCL_FMT_COO) {
        // nothing of a COO message is read before its header is checked
        if (o.bytes < kHeaderBytes) return SPCCL_ERR_CAPACITY;
        *out = Src{SRC_COO, DevOperand{p, p, o.bytes}};
    } else {
        return SPCCL_ERR_INVALID_ARG;
    }
    return SPCCL_OK;
}

uint64_t operand_extent(const spccl_operand_t& o) { return o.bytes; }

}  // namespace

extern "C" {

uint64_t spccl_num_tiles(uint64_t n) { return num_tiles(n); }

uint64_t spccl_pici_bytes(uint64_t n, int32_t dtype, uint64_t nnz) {
    return dtype_ok(dtype) ? pici_bytes(n, dtype, nnz) : 0;
}

uint64_t spccl_stream_bound(uint64_t n, int32_t dtype) {
    if (!dtype_ok(dtype)) return 0;
    const uint64_t p = pici_bytes(n, dtype, n), d = dense_msg_bytes(n, dtype);
    return p > d ? p : d;
}

uint64_t spccl_workspace_min_bytes(uint64_t n, int32_t dtype) {
    (void)dtype;
    return slots_offset(n);
}

uint64_t spccl_workspace_bytes(uint64_t n, int32_t dtype) {
    return value_slots_end(n, dtype) + num_parts(n) * kPartElems * 4ull;
}

uint64_t spccl_coo_bytes(int32_t dtype, uint64_t nnz) { return dtype_ok(dtype) ? coo_bytes(dtype, nnz) : 0; }

uint64_t spccl_message_bound(uint64_t n, int32_t dtype, int32_t fmt) {
    if (!dtype_ok(dtype)) return 0;
    const uint64_t d = dense_msg_bytes(n, dtype);
    uint64_t w;
    if (fmt == SPCCL_FMT_DENSE) w = d;
    else if (fmt == SPCCL_FMT_PICI) w = pici_bytes(n, dtype, n);
    else if (fmt == SPCCL_FMT_COO) w = coo_bytes(dtype, n);
    else return 0;
    return w > d ? w : d;
}

uint32_t spccl_set_single_pass_limit(uint32_t max_partitions) {
    return spccl::set_single_pass_max_parts(max_partitions);
}

spccl_status_t spccl_workspace_init(void* ws, uint64_t ws_bytes, void* stream) {
    if (!ws || !aligned16(ws) || ws_bytes < kWsFlagsOffset) return SPCCL_ERR_INVALID_ARG;
    return launch_fill_zero(ws, ws_bytes, as_stream(stream));
}

spccl_status_t spccl_compress(const void* dense, uint64_t n, int32_t dtype, void* out, uint64_t out_bytes,
                              void* ws, uint64_t ws_bytes, void* stream) {
    if (!dtype_ok(dtype)) return SPCCL_ERR_UNSUPPORTED;
    if (n >= (1ull << 32)) return SPCCL_ERR_UNSUPPORTED;
    if ((n && (!dense || !aligned_elem(dense, dtype))) || !out || !aligned16(out)) return SPCCL_ERR_INVALID_ARG;
    if (out_bytes < spccl_stream_bound(n, dtype)) return SPCCL_ERR_CAPACITY;
    if (overlaps(dense, n * elem_bytes(dtype), out, out_bytes)) return SPCCL_ERR_INVALID_ARG;
    spccl_status_t st = check_ws(ws, ws_bytes, spccl_workspace_min_bytes(n, dtype));
    if (st != SPCCL_OK) return st;
    PiciSinkArgs g{};
    g.slots = ws_bytes >= value_slots_end(n, dtype) ? static_cast<uint8_t*>(ws) + slots_offset(n) : nullptr;
    g.a = DevOperand{nullptr, static_cast<const uint8_t*>(dense), n * elem_bytes(dtype)};
    g.out = static_cast<uint8_t*>(out);
    g.n = n;
    g.T = num_tiles(n);
    g.nparts = (uint32_t)num_parts(n);
    g.epoch = next_epoch();
    g.ctrl = static_cast<WsCtrl*>(ws);
    g.flags = reinterpret_cast<uint64_t*>(static_cast<uint8_t*>(ws) + kWsFlagsOffset);
    return launch_to_pici_dt(dtype, SRC_DENSE, SRC_NONE, g, as_stream(stream));
}

namespace {
// The COO sink (two passes; needs the full workspace with its slots).
// A COO operand gets a tile index (k_coo_index) in the workspace when the
// workspace has room for it (spccl_workspace_min_bytes); otherwise its tiles
// search J for their entries.  The workspace has been checked.
spccl_status_t index_coo(Src& s, int which, uint64_t n, int32_t dtype, void* ws, uint64_t ws_bytes, hipStream_t hs) {
    if (s.kind != SRC_COO || n == 0 || ws_bytes < slots_offset(n)) return SPCCL_OK;
    uint64_t* idx = reinterpret_cast<uint64_t*>(static_cast<uint8_t*>(ws) + coo_index_offset(n, which));
    uint32_t epoch = next_epoch();
    if (epoch == 0) epoch = next_epoch();      // a zeroed workspace holds epoch-0 words
    s.dev.idx = idx;
    s.dev.idx_epoch = epoch;
    return launch_coo_index(s.dev.data, s.dev.cap, n, dtype, idx, epoch, static_cast<WsCtrl*>(ws), hs);
}

spccl_status_t run_coo_sink(Src sa, Src sb, uint8_t* out, uint64_t n, int32_t dtype, void* ws,
                            uint64_t ws_bytes, hipStream_t hs) {
    spccl_status_t st = check_ws(ws, ws_bytes, spccl_workspace_bytes(n, dtype));
    if (st != SPCCL_OK) return st;
    if ((st = index_coo(sa, 0, n, dtype, ws, ws_bytes, hs)) != SPCCL_OK) return st;
    if ((st = index_coo(sb, 1, n, dtype, ws, ws_bytes, hs)) != SPCCL_OK) return st;
    PiciSinkArgs g{};
    g.slots = static_cast<uint8_t*>(ws) + slots_offset(n);
    g.idx_slots = reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(ws) + value_slots_end(n, dtype));
    g.a = sa.dev;
    g.b = sb.dev;
    g.out = out;
    g.n = n;
    g.T = num_tiles(n);
    g.nparts = (uint32_t)num_parts(n);
    g.epoch = next_epoch();
    g.ctrl = static_cast<WsCtrl*>(ws);
    g.flags = reinterpret_cast<uint64_t*>(static_cast<uint8_t*>(ws) + kWsFlagsOffset);
    return launch_to_coo_dt(dtype, sa.kind, sb.kind, g, hs);
}
}  // namespace

spccl_status_t spccl_compress_coo(const void* dense, uint64_t n, int32_t dtype, void* out, uint64_t out_bytes,
                                  void* ws, uint64_t ws_bytes, void* stream) {
    if (!dtype_ok(dtype)) return SPCCL_ERR_UNSUPPORTED;
    if (n >= (1ull << 32)) return SPCCL_ERR_UNSUPPORTED;
    if ((n && (!dense || !aligned_elem(dense, dtype))) || !out || !aligned16(out)) return SPCCL_ERR_INVALID_ARG;
    if (out_bytes < spccl_message_bound(n, dtype, SPCCL_FMT_COO)) return SPCCL_ERR_CAPACITY;
    if (overlaps(dense, n * elem_bytes(dtype), out, out_bytes)) return SPCCL_ERR_INVALID_ARG;
    const Src sa{SRC_DENSE, DevOperand{nullptr, static_cast<const uint8_t*>(dense), n * elem_bytes(dtype)}};
    const Src sb{SRC_NONE, DevOperand{nullptr, nullptr, 0}};
    return run_coo_sink(sa, sb, static_cast<uint8_t*>(out), n, dtype, ws, ws_bytes, as_stream(stream));
}

spccl_status_t spccl_encode_dense(const void* dense, uint64_t n, int32_t dtype, void* out, uint64_t out_bytes,
                                  void* stream) {
    if (!dtype_ok(dtype)) return SPCCL_ERR_UNSUPPORTED;
    if (n >= (1ull << 32)) return SPCCL_ERR_UNSUPPORTED;
    if ((n && (!dense || !aligned_elem(dense, dtype))) || !out || !aligned16(out)) return SPCCL_ERR_INVALID_ARG;
    if (out_bytes < dense_msg_bytes(n, dtype)) return SPCCL_ERR_CAPACITY;
    if (overlaps(dense, n * elem_bytes(dtype), out, out_bytes)) return SPCCL_ERR_INVALID_ARG;
    return launch_encode_dense_dt(dtype, static_cast<const uint8_t*>(dense), static_cast<uint8_t*>(out), n,
                                  as_stream(stream));
}

spccl_status_t spccl_gather_expand(const spccl_operand_t* parts, int32_t P, uint64_t n_per_part, int32_t dtype,
                                   void* dense_out, uint64_t out_bytes, void* ws, uint64_t ws_bytes,
                                   void* stream) {
    if (!dtype_ok(dtype)) return SPCCL_ERR_UNSUPPORTED;
    if (n_per_part >= (1ull << 32)) return SPCCL_ERR_UNSUPPORTED;
    if (!parts || P < 0) return SPCCL_ERR_INVALID_ARG;
    if (P == 0) return SPCCL_OK;
    const uint64_t s = elem_bytes(dtype);
    if (!dense_out || !aligned_elem(dense_out, dtype)) return SPCCL_ERR_INVALID_ARG;
    if (out_bytes < (uint64_t)P * n_per_part * s) return SPCCL_ERR_CAPACITY;
    spccl_status_t st = check_ws(ws, ws_bytes, kWsFlagsOffset);
    if (st != SPCCL_OK) return st;
    if (n_per_part == 0) return SPCCL_OK;
    // every part is checked before the first launch: a bad part anywhere
    // returns its error with nothing launched, however many launches the
    // parts take
    for (int32_t q = 0; q < P; q++) {
        const spccl_operand_t& o = parts[q];
        if (!o.ptr || (o.kind == SPCCL_ARRAY ? !aligned_elem(o.ptr, dtype) : !aligned16(o.ptr)))
            return SPCCL_ERR_INVALID_ARG;
        if (o.kind == SPCCL_ARRAY) {
            if (o.bytes < n_per_part * s) return SPCCL_ERR_CAPACITY;
        } else if (o.kind == SPCCL_STREAM) {
            if (o.bytes < kHeaderBytes) return SPCCL_ERR_CAPACITY;
        } else {
            return SPCCL_ERR_INVALID_ARG;
        }
        if (overlaps(o.ptr, o.bytes, dense_out, out_bytes)) return SPCCL_ERR_INVALID_ARG;
    }
    GatherArgs g{};
    g.n = n_per_part;
    g.T = num_tiles(n_per_part);
    g.ctrl = static_cast<WsCtrl*>(ws);
    for (int32_t q0 = 0; q0 < P; q0 += kMaxGatherParts) {
        const int cnt = (P - q0) < kMaxGatherParts ? (P - q0) : kMaxGatherParts;
        for (int k = 0; k < cnt; k++) {
            const spccl_operand_t& o = parts[q0 + k];
            const uint8_t* p = static_cast<const uint8_t*>(o.ptr);
            g.part[k] = o.kind == SPCCL_ARRAY ? DevOperand{nullptr, p, o.bytes} : DevOperand{p, p, o.bytes};
        }
        g.out = static_cast<uint8_t*>(dense_out) + (uint64_t)q0 * n_per_part * s;
        st = launch_gather_dt(dtype, g, cnt, as_stream(stream));
        if (st != SPCCL_OK) return st;
    }
    return SPCCL_OK;
}

spccl_status_t spccl_decompress(const void* in, uint64_t in_bytes, void* dense, uint64_t n, int32_t dtype,
                                void* ws, uint64_t ws_bytes, void* stream) {
    spccl_operand_t part{SPCCL_STREAM, SPCCL_FMT_PICI, const_cast<void*>(in), in_bytes};
    return spccl_gather_expand(&part, 1, n, dtype, dense, n * (dtype == kBF16 ? 2u : 4u), ws, ws_bytes, stream);
}

spccl_status_t spccl_reduce(spccl_operand_t a, spccl_operand_t b, spccl_operand_t out, uint64_t n, int32_t dtype,
                            void* ws, uint64_t ws_bytes, void* stream) {
    if (!dtype_ok(dtype)) return SPCCL_ERR_UNSUPPORTED;
    if (n >= (1ull << 32)) return SPCCL_ERR_UNSUPPORTED;
    const uint64_t s = elem_bytes(dtype);
    Src sa{}, sb{};
    spccl_status_t st = decode_input(a, n, dtype, &sa);
    if (st != SPCCL_OK) return st;
    st = decode_input(b, n, dtype, &sb);
    if (st != SPCCL_OK) return st;
    if (!out.ptr || (out.kind == SPCCL_ARRAY ? !aligned_elem(out.ptr, dtype) : !aligned16(out.ptr)))
        return SPCCL_ERR_INVALID_ARG;
    // aliasing: only ARRAY out == ARRAY input exactly (in-place accumulation)
    for (const spccl_operand_t* in : {&a, &b}) {
        if (!overlaps(out.ptr, operand_extent(out), in->ptr, operand_extent(*in))) continue;
        const bool inplace = out.kind == SPCCL_ARRAY && in->kind == SPCCL_ARRAY && out.ptr == in->ptr;
        if (!inplace) return SPCCL_ERR_INVALID_ARG;
    }
    hipStream_t hs = as_stream(stream);
    WsCtrl* ctrl = static_cast<WsCtrl*>(ws);
    // Pici and COO do not meet in one call: a COO operand combines with dense
    // operands or another COO operand, into a dense or COO result
    const bool any_coo = sa.kind == SRC_COO || sb.kind == SRC_COO;
    const bool any_pici = sa.kind == SRC_PICI || sb.kind == SRC_PICI;
    const bool out_pici = out.kind == SPCCL_STREAM && out.fmt == SPCCL_FMT_PICI;
    const bool out_coo = out.kind == SPCCL_STREAM && out.fmt == SPCCL_FMT_COO;
    if ((any_coo && (any_pici || out_pici)) || (out_coo && any_pici)) return SPCCL_ERR_UNSUPPORTED;
    if (out_coo) {
        if (out.bytes < spccl_message_bound(n, dtype, SPCCL_FMT_COO)) return SPCCL_ERR_CAPACITY;
        return run_coo_sink(sa, sb, static_cast<uint8_t*>(out.ptr), n, dtype, ws, ws_bytes, hs);
    }
    if (out.kind == SPCCL_STREAM && out.fmt == SPCCL_FMT_PICI) {
        if (out.bytes < spccl_stream_bound(n, dtype)) return SPCCL_ERR_CAPACITY;
        st = check_ws(ws, ws_bytes, spccl_workspace_min_bytes(n, dtype));
        if (st != SPCCL_OK) return st;
        PiciSinkArgs g{};
        g.slots = ws_bytes >= value_slots_end(n, dtype) ? static_cast<uint8_t*>(ws) + slots_offset(n) : nullptr;
        g.a = sa.dev;
        g.b = sb.dev;
        g.out = static_cast<uint8_t*>(out.ptr);
        g.n = n;
        g.T = num_tiles(n);
        g.nparts = (uint32_t)num_parts(n);
        g.epoch = next_epoch();
        g.ctrl = ctrl;
        g.flags = reinterpret_cast<uint64_t*>(static_cast<uint8_t*>(ws) + kWsFlagsOffset);
        return launch_to_pici_dt(dtype, sa.kind, sb.kind, g, hs);
    }
    uint8_t* out_hdr = nullptr;
    uint8_t* out_data = static_cast<uint8_t*>(out.ptr);
    if (out.kind == SPCCL_STREAM) {
        if (out.fmt != SPCCL_FMT_DENSE) return SPCCL_ERR_INVALID_ARG;
        if (out.bytes < dense_msg_bytes(n, dtype)) return SPCCL_ERR_CAPACITY;
        out_hdr = out_data;
        out_data += kHeaderBytes;
    } else if (out.kind == SPCCL_ARRAY) {
        if (out.bytes < n * s) return SPCCL_ERR_CAPACITY;
    } else {
        return SPCCL_ERR_INVALID_ARG;
    }
    st = check_ws(ws, ws_bytes, kWsFlagsOffset);
    if (st != SPCCL_OK) return st;
    if (sa.kind == SRC_DENSE && sb.kind == SRC_DENSE)
        return launch_dense_dense_dt(dtype, sa.dev.hdr, sa.dev.data, sa.dev.cap, sb.dev.hdr, sb.dev.data,
                                     sb.dev.cap, out_hdr, out_data, n, ctrl, hs);
    if (n == 0 && !out_hdr) return SPCCL_OK;
    if ((st = index_coo(sa, 0, n, dtype, ws, ws_bytes, hs)) != SPCCL_OK) return st;
    if ((st = index_coo(sb, 1, n, dtype, ws, ws_bytes, hs)) != SPCCL_OK) return st;
    DenseSinkArgs g{};
    g.a = sa.dev;
    g.b = sb.dev;
    g.out_hdr = out_hdr;
    g.out = out_data;
    g.n = n;
    g.T = num_tiles(n);
    g.ctrl = ctrl;
    return launch_to_dense_dt(dtype, sa.kind, sb.kind, g, hs);
}

spccl_status_t spccl_copy_message(const void* src, uint64_t src_bytes, void* dst, uint64_t dst_bytes, void* ws,
                                  uint64_t ws_bytes, void* stream) {
    if (!src || !dst || !aligned16(src) || !aligned16(dst)) return SPCCL_ERR_INVALID_ARG;
    if (src_bytes < kHeaderBytes) return SPCCL_ERR_CAPACITY;
    if (overlaps(src, src_bytes, dst, dst_bytes)) return SPCCL_ERR_INVALID_ARG;
    spccl_status_t st = check_ws(ws, ws_bytes, kWsFlagsOffset);
    if (st != SPCCL_OK) return st;
    return launch_copy_message(static_cast<const uint8_t*>(src), src_bytes, static_cast<uint8_t*>(dst), dst_bytes,
                               static_cast<WsCtrl*>(ws), as_stream(stream));
}

/* ---- sliced streams ---------------------------------------------------------- */

uint64_t spccl_slice_count(uint64_t n) { return num_slices(n); }

uint64_t spccl_slice_bytes(int32_t dtype) { return dtype_ok(dtype) ? slice_slot_bytes(dtype) : 0; }

namespace {

// Common checks of the sliced entry points: a dense array (element-aligned,
// n elements) and sliced streams (16-byte aligned, every slot present).
spccl_status_t check_sliced_args(uint64_t n, int32_t dtype, void* ws, uint64_t ws_bytes) {
    if (!dtype_ok(dtype)) return SPCCL_ERR_UNSUPPORTED;
    if (n >= (1ull << 32)) return SPCCL_ERR_UNSUPPORTED;
    return check_ws(ws, ws_bytes, kWsFlagsOffset);
}

spccl_status_t check_dense_arg(const void* p, uint64_t bytes, uint64_t n, int32_t dtype) {
    if (!p || !aligned_elem(p, dtype)) return SPCCL_ERR_INVALID_ARG;
    return bytes < n * elem_bytes(dtype) ? SPCCL_ERR_CAPACITY : SPCCL_OK;
}

spccl_status_t check_sliced_arg(const void* p, uint64_t bytes, uint64_t n, int32_t dtype) {
    if (!p || !aligned16(p)) return SPCCL_ERR_INVALID_ARG;
    return bytes < num_slices(n) * slice_slot_bytes(dtype) ? SPCCL_ERR_CAPACITY : SPCCL_OK;
}

}  // namespace

spccl_status_t spccl_compress_sliced(const void* dense, uint64_t n, int32_t dtype, double dense_thresh, void* out,
                                     uint64_t out_bytes, void* ws, uint64_t ws_bytes, void* stream) {
    spccl_status_t st = check_sliced_args(n, dtype, ws, ws_bytes);
    if (st == SPCCL_OK) st = check_dense_arg(dense, n * elem_bytes(dtype), n, dtype);
    if (st == SPCCL_OK) st = check_sliced_arg(out, out_bytes, n, dtype);
    if (st != SPCCL_OK) return st;
    if (overlaps(dense, n * elem_bytes(dtype), out, out_bytes)) return SPCCL_ERR_INVALID_ARG;
    if (n == 0) return SPCCL_OK;
    SlicedArgs g{static_cast<const uint8_t*>(dense), nullptr, static_cast<uint8_t*>(out), n, slice_slot_bytes(dtype),
                 dense_thresh, static_cast<WsCtrl*>(ws)};
    return launch_sliced_dt(dtype, g, kSlicedCompress, as_stream(stream));
}

spccl_status_t spccl_decompress_sliced(const void* in, uint64_t in_bytes, void* dense, uint64_t n, int32_t dtype,
                                       void* ws, uint64_t ws_bytes, void* stream) {
    spccl_status_t st = check_sliced_args(n, dtype, ws, ws_bytes);
    if (st == SPCCL_OK) st = check_sliced_arg(in, in_bytes, n, dtype);
    if (st == SPCCL_OK) st = check_dense_arg(dense, n * elem_bytes(dtype), n, dtype);
    if (st != SPCCL_OK) return st;
    if (overlaps(in, in_bytes, dense, n * elem_bytes(dtype))) return SPCCL_ERR_INVALID_ARG;
    if (n == 0) return SPCCL_OK;
    SlicedArgs g{static_cast<const uint8_t*>(in), nullptr, static_cast<uint8_t*>(dense), n, slice_slot_bytes(dtype),
                 0.0, static_cast<WsCtrl*>(ws)};
    return launch_sliced_dt(dtype, g, kSlicedExpand, as_stream(stream));
}

spccl_status_t spccl_reduce_sliced(const void* a, const void* b, uint64_t b_bytes, void* out, uint64_t out_bytes,
                                   int32_t out_sliced, double dense_thresh, uint64_t n, int32_t dtype, void* ws,
                                   uint64_t ws_bytes, void* stream) {
    spccl_status_t st = check_sliced_args(n, dtype, ws, ws_bytes);
    if (st == SPCCL_OK) st = check_dense_arg(a, n * elem_bytes(dtype), n, dtype);
    if (st == SPCCL_OK) st = check_sliced_arg(b, b_bytes, n, dtype);
    if (st == SPCCL_OK)
        st = out_sliced ? check_sliced_arg(out, out_bytes, n, dtype) : check_dense_arg(out, out_bytes, n, dtype);
    if (st != SPCCL_OK) return st;
    const uint64_t ab = n * elem_bytes(dtype);
    // a dense output may overwrite a in place (each element is read before it is written, by the same lane)
    if (overlaps(b, b_bytes, out, out_bytes) || overlaps(a, ab, b, b_bytes)) return SPCCL_ERR_INVALID_ARG;
    if (out_sliced ? overlaps(a, ab, out, out_bytes) : (overlaps(a, ab, out, out_bytes) && a != out))
        return SPCCL_ERR_INVALID_ARG;
    if (n == 0) return SPCCL_OK;
    SlicedArgs g{static_cast<const uint8_t*>(a), static_cast<const uint8_t*>(b), static_cast<uint8_t*>(out), n,
                 slice_slot_bytes(dtype), dense_thresh, static_cast<WsCtrl*>(ws)};
    return launch_sliced_dt(dtype, g, out_sliced ? kSlicedReduceToSliced : kSlicedReduceToDense, as_stream(stream));
}

uint64_t spccl_slice_tracker_bytes(uint64_t n) { return 16ull * num_slices(n); }

namespace {
spccl_status_t check_tracker(const double* track, uint64_t track_bytes, uint64_t n) {
    if (!track || (reinterpret_cast<uintptr_t>(track) & 7u)) return SPCCL_ERR_INVALID_ARG;
    return track_bytes < 16ull * num_slices(n) ? SPCCL_ERR_CAPACITY : SPCCL_OK;
}
}  // namespace

spccl_status_t spccl_compress_sliced_tracked(const void* dense, uint64_t n, int32_t dtype, double tau, void* out,
                                             uint64_t out_bytes, double* tracker, uint64_t tracker_bytes,
                                             uint8_t* fmt_out, void* ws, uint64_t ws_bytes, void* stream) {
    spccl_status_t st = check_sliced_args(n, dtype, ws, ws_bytes);
    if (st == SPCCL_OK) st = check_dense_arg(dense, n * elem_bytes(dtype), n, dtype);
    if (st == SPCCL_OK) st = check_sliced_arg(out, out_bytes, n, dtype);
    if (st == SPCCL_OK) st = check_tracker(tracker, tracker_bytes, n);
    if (st != SPCCL_OK) return st;
    if (overlaps(dense, n * elem_bytes(dtype), out, out_bytes) || overlaps(tracker, tracker_bytes, out, out_bytes))
        return SPCCL_ERR_INVALID_ARG;
    if (n == 0) return SPCCL_OK;
    SlicedArgs g{static_cast<const uint8_t*>(dense), nullptr, static_cast<uint8_t*>(out), n, slice_slot_bytes(dtype),
                 tau, static_cast<WsCtrl*>(ws), tracker, 0, fmt_out};
    return launch_sliced_dt(dtype, g, kSlicedCompress, as_stream(stream));
}

spccl_status_t spccl_reduce_sliced_tracked(const void* a, const void* b, uint64_t b_bytes, void* out,
                                           uint64_t out_bytes, double tau, double* tracker, uint64_t tracker_bytes,
                                           uint8_t* fmt_out, uint64_t n, int32_t dtype, void* ws, uint64_t ws_bytes,
                                           void* stream) {
    spccl_status_t st = check_sliced_args(n, dtype, ws, ws_bytes);
    if (st == SPCCL_OK) st = check_dense_arg(a, n * elem_bytes(dtype), n, dtype);
    if (st == SPCCL_OK) st = check_sliced_arg(b, b_bytes, n, dtype);
    if (st == SPCCL_OK) st = check_sliced_arg(out, out_bytes, n, dtype);
    if (st == SPCCL_OK) st = check_tracker(tracker, tracker_bytes, n);
    if (st != SPCCL_OK) return st;
    const uint64_t ab = n * elem_bytes(dtype);
    if (overlaps(b, b_bytes, out, out_bytes) || overlaps(a, ab, b, b_bytes) || overlaps(a, ab, out, out_bytes) ||
        overlaps(tracker, tracker_bytes, out, out_bytes))
        return SPCCL_ERR_INVALID_ARG;
    if (n == 0) return SPCCL_OK;
    SlicedArgs g{static_cast<const uint8_t*>(a), static_cast<const uint8_t*>(b), static_cast<uint8_t*>(out), n,
                 slice_slot_bytes(dtype), tau, static_cast<WsCtrl*>(ws), tracker, 1, fmt_out};
    return launch_sliced_dt(dtype, g, kSlicedReduceToSliced, as_stream(stream));
}

spccl_status_t spccl_copy_sliced(const void* src, uint64_t src_bytes, void* dst, uint64_t dst_bytes, uint64_t n,
                                 int32_t dtype, void* ws, uint64_t ws_bytes, void* stream) {
    spccl_status_t st = check_sliced_args(n, dtype, ws, ws_bytes);
    if (st == SPCCL_OK) st = check_sliced_arg(src, src_bytes, n, dtype);
    if (st == SPCCL_OK) st = check_sliced_arg(dst, dst_bytes, n, dtype);
    if (st != SPCCL_OK) return st;
    if (overlaps(src, src_bytes, dst, dst_bytes)) return SPCCL_ERR_INVALID_ARG;
    if (n == 0) return SPCCL_OK;
    SlicedArgs g{static_cast<const uint8_t*>(src), nullptr, static_cast<uint8_t*>(dst), n, slice_slot_bytes(dtype),
                 0.0, static_cast<WsCtrl*>(ws)};
    return launch_copy_sliced(g, as_stream(stream));
}

spccl_status_t spccl_read_header(const void* msg, spccl_header_t* host_out, void* stream) {
    if (!msg || !host_out) return SPCCL_ERR_INVALID_ARG;
    hipStream_t hs = as_stream(stream);
    if (hipMemcpyAsync(host_out, msg, sizeof(spccl_header_t), hipMemcpyDeviceToHost, hs) != hipSuccess)
        return SPCCL_ERR_HIP;
    return hipStreamSynchronize(hs) == hipSuccess ? SPCCL_OK : SPCCL_ERR_HIP;
}

spccl_status_t spccl_read_status(void* ws, int32_t clear, void* stream) {
    if (!ws || !aligned16(ws)) return SPCCL_ERR_INVALID_ARG;
    hipStream_t hs = as_stream(stream);
    uint32_t v = 0;
    if (hipMemcpyAsync(&v, ws, sizeof(v), hipMemcpyDeviceToHost, hs) != hipSuccess) return SPCCL_ERR_HIP;
    if (hipStreamSynchronize(hs) != hipSuccess) return SPCCL_ERR_HIP;
    if (clear && v != 0) {
        if (launch_fill_zero(ws, sizeof(uint32_t), hs) != SPCCL_OK) return SPCCL_ERR_HIP;
        if (hipStreamSynchronize(hs) != hipSuccess) return SPCCL_ERR_HIP;
    }
    return static_cast<spccl_status_t>(v);
}

const char* spccl_status_string(spccl_status_t s) {
    switch (s) {
        case SPCCL_OK: return "ok";
        case SPCCL_ERR_INVALID_ARG: return "invalid argument";
        case SPCCL_ERR_CAPACITY: return "buffer capacity too small";
        case SPCCL_ERR_UNSUPPORTED: return "unsupported dtype or size";
        case SPCCL_ERR_CORRUPT_STREAM: return "corrupt message";
        case SPCCL_ERR_WORKSPACE: return "workspace too small";
        case SPCCL_ERR_HIP: return "HIP runtime error";
        case SPCCL_ERR_TIMEOUT: return "device wait exceeded its spin limit";
    }
    return "unknown status";
}

}  // extern "C"
