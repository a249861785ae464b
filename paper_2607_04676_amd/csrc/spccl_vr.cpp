// Ring collectives over P virtual ranks held in one GPU's memory (Sec. IV).
//
// Sparse sends are Pici messages or, with policy.sparse_fmt = COO, COO
// messages (the paper runs both, Sec. IV-D).  Each rank's send / receive
// buffers are regions of one scratch allocation;
// a "send" is a device-side copy of the message (its size is read from the
// header on the device).  Format decisions are made on the host, per sending
// rank, from the nonzero counts the compressing kernels write into the
// message headers: one stream synchronization per ring step reads all P
// headers with a single strided copy.
//
// Decision rule (Sec. IV-C):
//   step 0      compress the first chunk, sigma0 = sigma_prev = measured;
//               send dense iff sigma0 <= tau(link)
//   step s > 0  est = sigma_prev * sigma0 (Eq. 7); if est <= tau(link),
//               reduce to a dense message and track est; otherwise reduce and
//               compress in one pass and track the measured sparsity
//   all-reduce  at the reduce-scatter -> all-gather transition each rank
//               gathers densely iff sigma_prev * sigma0 <= ag_thresh
// tau(link) is inter_thresh on a link r -> r+1 that leaves a node
// ((r+1) % ranks_per_node == 0) and intra_thresh otherwise.
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <string.h>

#include <vector>

#include "spccl_internal.h"
#include "../../include/spccl.h"

using namespace spccl;

namespace spccl {
spccl_status_t launch_sliced_batch_dt(int dtype, const SlicedBatch& b, uint32_t ranks, int op, hipStream_t st);
spccl_status_t launch_copy_sliced_batch(const SlicedBatch& b, uint32_t ranks, hipStream_t st);
spccl_status_t launch_to_pici_rb_dt(int dtype, int sa, int sb, const PiciSinkArgs& g, const RankBatch& rb,
                                    uint32_t ranks, hipStream_t st);
spccl_status_t launch_to_dense_rb_dt(int dtype, int sa, int sb, const DenseSinkArgs& g, const RankBatch& rb,
                                     uint32_t ranks, hipStream_t st);
spccl_status_t launch_copy_message_rb(uint64_t src_cap, uint64_t dst_cap, WsCtrl* ctrl, const RankBatch& rb,
                                      uint32_t ranks, hipStream_t st);
spccl_status_t launch_encode_dense_rb_dt(int dtype, uint64_t n, const RankBatch& rb, uint32_t ranks, hipStream_t st);
spccl_status_t launch_gather_rb_dt(int dtype, const DevOperand& part, uint64_t n, WsCtrl* ctrl, const RankBatch& rb,
                                   uint32_t ranks, hipStream_t st);
spccl_status_t launch_fill_zero(void* p, uint64_t bytes, hipStream_t st);
spccl_status_t launch_ring_decide(const RingArgs& a, hipStream_t st);
}  // namespace spccl

namespace {

constexpr uint64_t kAlign = 256;
inline uint64_t round_up(uint64_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
inline bool overlaps(const void* a, uint64_t an, const void* b, uint64_t bn) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return an && bn && x < y + bn && y < x + an;
}
inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// Scratch of the canonical collectives: one full workspace (its control block
// holds the status word every launch of the call reports to; the per-rank
// calls of COO sends use the rest), then for the batched Pici launches one
// region of look-back words and one of value slots per rank, then 3 * P
// message buffers.
struct Layout {
    uint8_t* ws;
    uint64_t ws_bytes;
    uint8_t* flags;             // P regions of look-back words (zeroed at the start of a call)
    uint64_t flag_bytes;        // per rank
    uint8_t* vslots;            // P regions of value slots
    uint64_t vslot_bytes;       // per rank
    uint64_t slot_bytes;        // capacity of one message buffer
    uint8_t* slots;             // 3 * P message buffers
    RingRank* rr;               // per rank: the device-side decision state
    spccl_trace_t* dtrace;      // the trace, written on the device
    uint8_t* slot(int which, int r, int P) const { return slots + ((uint64_t)which * P + r) * slot_bytes; }
    uint8_t* rank_flags(int r) const { return flags + (uint64_t)r * flag_bytes; }
    uint8_t* rank_slots(int r) const { return vslots + (uint64_t)r * vslot_bytes; }
};

// every message buffer holds the worst case of any format: COO's for long
// messages, Pici's (the column words and offsets of a whole tile) for short ones
uint64_t slot_need(uint64_t msg_elems, int32_t dtype) {
    const uint64_t c = spccl_message_bound(msg_elems, dtype, SPCCL_FMT_COO), p = spccl_stream_bound(msg_elems, dtype);
    return round_up(c > p ? c : p);
}

Layout carve(void* scratch, int32_t P, uint64_t msg_elems, int32_t dtype) {
    Layout L;
    L.ws = static_cast<uint8_t*>(scratch);
    L.ws_bytes = round_up(spccl_workspace_bytes(msg_elems, dtype));
    L.flags = L.ws + L.ws_bytes;
    L.flag_bytes = round_up(8ull * flag_words(msg_elems));
    L.vslots = L.flags + (uint64_t)P * L.flag_bytes;
    L.vslot_bytes = round_up(num_parts(msg_elems) * kPartElems * elem_bytes(dtype));
    L.slot_bytes = slot_need(msg_elems, dtype);
    L.slots = L.vslots + (uint64_t)P * L.vslot_bytes;
    L.rr = reinterpret_cast<RingRank*>(L.slots + 3ull * (uint64_t)P * L.slot_bytes);
    L.dtrace = reinterpret_cast<spccl_trace_t*>(reinterpret_cast<uint8_t*>(L.rr) + round_up(sizeof(RingRank) * P));
    return L;
}

uint64_t scratch_need(int32_t P, uint64_t msg_elems, int32_t dtype) {
    const Layout L = carve(nullptr, P, msg_elems, dtype);
    const uint64_t trace_entries = (uint64_t)P * (uint64_t)(P - 1) + (uint64_t)P;
    return (uint64_t)(reinterpret_cast<uint8_t*>(L.dtrace) - L.ws) + round_up(sizeof(spccl_trace_t) * trace_entries);
}

// Zero the parts of the scratch that must start clear: the workspace's
// control block, look-back words and tile indexes, and every rank's
// look-back words (the value slots and message buffers are written before
// they are read).
spccl_status_t init_scratch(const Layout& L, int32_t P, uint64_t msg_elems, int32_t dtype, hipStream_t st) {
    spccl_status_t s1 = launch_fill_zero(L.ws, spccl_workspace_min_bytes(msg_elems, dtype), st);
    if (s1 != SPCCL_OK) return s1;
    return launch_fill_zero(L.flags, (uint64_t)P * L.flag_bytes, st);
}

double link_tau(const spccl_policy_t& pol, int r, int P) {
    const int rpn = pol.ranks_per_node > 0 ? pol.ranks_per_node : P;
    return ((r + 1) % rpn == 0 && rpn < P) ? pol.inter_thresh : pol.intra_thresh;
}

bool send_dense(const spccl_policy_t& pol, double sigma, double tau) {
    if (pol.adaptive == 0) return false;
    if (pol.adaptive == 2) return true;
    return sigma <= tau;
}

double sparsity(uint64_t m, uint64_t nnz) { return m == 0 ? 1.0 : (double)(m - nnz) / (double)m; }

// Read the headers of message slot `which` of all P ranks (one strided copy).
spccl_status_t read_headers(const Layout& L, int which, int P, std::vector<spccl_header_t>& h, hipStream_t st) {
    h.resize(P);
    if (hipMemcpy2DAsync(h.data(), sizeof(spccl_header_t), L.slot(which, 0, P), L.slot_bytes, sizeof(spccl_header_t),
                         P, hipMemcpyDeviceToHost, st) != hipSuccess)
        return SPCCL_ERR_HIP;
    return hipStreamSynchronize(st) == hipSuccess ? SPCCL_OK : SPCCL_ERR_HIP;
}

void put_trace(spccl_trace_t* tr, int idx, int step, int rank, int fmt, int measured, uint64_t bytes, uint64_t nnz,
               double sigma) {
    if (!tr) return;
    tr[idx] = spccl_trace_t{step, rank, fmt, measured, bytes, nnz, sigma};
}

spccl_operand_t arr(const void* p, uint64_t bytes) {
    return spccl_operand_t{SPCCL_ARRAY, 0, const_cast<void*>(p), bytes};
}
spccl_operand_t msg(void* p, int fmt, uint64_t bytes) { return spccl_operand_t{SPCCL_STREAM, fmt, p, bytes}; }

// the sparse encoding of the collective (Pici, or COO as in Sec. IV-D)
spccl_status_t compress_fmt(int fmt, const void* dense, uint64_t m, int dtype, const Layout& L, uint8_t* out,
                            hipStream_t st) {
    if (fmt == SPCCL_FMT_COO) return spccl_compress_coo(dense, m, dtype, out, L.slot_bytes, L.ws, L.ws_bytes, st);
    return spccl_compress(dense, m, dtype, out, L.slot_bytes, L.ws, L.ws_bytes, st);
}

const spccl_policy_t kDefaultPolicy{0.6, 0.5, 0.1, 0, 1, SPCCL_FMT_PICI};

bool policy_ok(const spccl_policy_t& pol) {
    return (pol.sparse_fmt == SPCCL_FMT_PICI || pol.sparse_fmt == SPCCL_FMT_COO) && pol.adaptive >= 0 &&
           pol.adaptive <= 2;
}

#define SPCCL_TRY(x)                               \
    do {                                           \
        spccl_status_t st_ = (x);                  \
        if (st_ != SPCCL_OK) return st_;           \
    } while (0)

// ---- batched ring steps, decided on the device (Pici sends) --------------
// Every ring step launches each kernel once for all ranks that may take that
// path (grid y = rank, up to kMaxBatchRanks per launch): the P reductions,
// sends and expansions of a step are independent of each other.  The format
// decisions are made on the device between the launches (k_ring_decide), and
// each rank's blocks skip the paths its decision rules out, so the host
// enqueues the whole collective and synchronizes once, at the end.

struct RankPtrs {
    const uint8_t* a;
    const uint8_t* b;
    uint8_t* out;
};

// The formats a batched launch is for (checked per rank on the device).
struct Gate {
    const RingRank* rr;       // null: every rank takes part
    int in_fmt, out_fmt;      // -1: any
};
constexpr Gate kNoGate{nullptr, -1, -1};

// launch(rb, count) for the given ranks in batches of up to kMaxBatchRanks,
// each rank's pointers from ptrs(rank) and its own look-back words and slots.
template <class Ptrs, class Launch>
spccl_status_t batched(const Layout& L, const std::vector<int>& ranks, Gate gate, Ptrs ptrs, Launch launch) {
    for (size_t i = 0; i < ranks.size(); i += kMaxBatchRanks) {
        const uint32_t cnt = (uint32_t)(ranks.size() - i < (size_t)kMaxBatchRanks ? ranks.size() - i : kMaxBatchRanks);
        RankBatch rb{};
        rb.gate = gate.rr;
        rb.gate_in = gate.in_fmt;
        rb.gate_out = gate.out_fmt;
        for (uint32_t j = 0; j < cnt; j++) {
            const int r = ranks[i + j];
            const RankPtrs q = ptrs(r);
            rb.a[j] = q.a;
            rb.b[j] = q.b;
            rb.out[j] = q.out;
            rb.flags[j] = L.rank_flags(r);
            rb.slots[j] = L.rank_slots(r);
            rb.rank[j] = r;
        }
        SPCCL_TRY(launch(rb, cnt));
    }
    return SPCCL_OK;
}

// an operand whose pointer comes from the batch: an array, a Pici (or any)
// message, a dense message
DevOperand arr_op(uint64_t bytes) { return DevOperand{nullptr, nullptr, bytes}; }
DevOperand msg_op(const Layout& L) { return DevOperand{L.slots, L.slots, L.slot_bytes}; }
DevOperand dense_msg_op(const Layout& L) { return DevOperand{L.slots, L.slots + kHeaderBytes, L.slot_bytes}; }

PiciSinkArgs sink_args(const Layout& L, uint64_t m, DevOperand a, DevOperand b) {
    PiciSinkArgs g{};
    g.a = a;
    g.b = b;
    g.n = m;
    g.T = num_tiles(m);
    g.nparts = (uint32_t)num_parts(m);
    g.epoch = next_epoch();
    g.ctrl = reinterpret_cast<WsCtrl*>(L.ws);
    g.slots = L.vslots;           // each rank's own, from the batch
    g.flags = reinterpret_cast<uint64_t*>(L.flags);
    return g;
}

DenseSinkArgs dense_args(const Layout& L, uint64_t m, DevOperand a, DevOperand b, bool out_msg) {
    DenseSinkArgs g{};
    g.a = a;
    g.b = b;
    g.out_hdr = out_msg ? L.slots : nullptr;
    g.out = out_msg ? L.slots + kHeaderBytes : L.slots;
    g.n = m;
    g.T = num_tiles(m);
    g.ctrl = reinterpret_cast<WsCtrl*>(L.ws);
    return g;
}

RingArgs ring_args(const Layout& L, int P, uint64_t m, int dtype, const spccl_policy_t& pol, int mode, int step) {
    RingArgs a{};
    a.rr = L.rr;
    a.trace = L.dtrace;
    a.slots0 = L.slot(0, 0, P);
    a.slot_bytes = L.slot_bytes;
    a.m = m;
    a.P = P;
    a.step = step;
    a.mode = mode;
    a.dtype = dtype;
    a.intra = pol.intra_thresh;
    a.inter = pol.inter_thresh;
    a.ag = pol.ag_thresh;
    a.ranks_per_node = pol.ranks_per_node;
    a.adaptive = pol.adaptive;
    return a;
}

// src(r) (m elements) into out(r) for the ranks whose decision is Pici
// (compressed) and dense (a dense message); gated on the device unless gate
// is kNoGate, when every rank compresses.
template <class Src, class Out>
spccl_status_t batched_encode(const Layout& L, const std::vector<int>& ranks, Gate gate, bool with_dense, uint64_t m,
                              int32_t dtype, Src src, Out out, hipStream_t st) {
    const uint64_t s = elem_bytes(dtype);
    auto ptrs = [&](int r) { return RankPtrs{src(r), nullptr, out(r)}; };
    const PiciSinkArgs g = sink_args(L, m, arr_op(m * s), DevOperand{});
    Gate gp = gate;
    if (gp.rr) gp.out_fmt = SPCCL_FMT_PICI;
    SPCCL_TRY(batched(L, ranks, gp, ptrs, [&](const RankBatch& rb, uint32_t c) {
        return launch_to_pici_rb_dt(dtype, SRC_DENSE, SRC_NONE, g, rb, c, st);
    }));
    if (with_dense && gate.rr) {
        Gate gd = gate;
        gd.out_fmt = SPCCL_FMT_DENSE;
        SPCCL_TRY(batched(L, ranks, gd, ptrs, [&](const RankBatch& rb, uint32_t c) {
            return launch_encode_dense_rb_dt(dtype, m, rb, c, st);
        }));
    }
    return SPCCL_OK;
}

// The reduce-scatter with Pici sends and device-side decisions: the same
// messages, results and trace (in L.dtrace) as ring_rs.
spccl_status_t ring_rs_dev(void* const* send, void* const* out, int P, uint64_t n, int dtype,
                           const spccl_policy_t& pol, const Layout& L, hipStream_t st) {
    const uint64_t m = n / (uint64_t)P, s = elem_bytes(dtype);
    auto chunk = [&](int r, int c) { return static_cast<const uint8_t*>(send[r]) + (uint64_t)c * m * s; };
    std::vector<int> all(P);
    for (int r = 0; r < P; r++) all[r] = r;
    WsCtrl* ctrl = reinterpret_cast<WsCtrl*>(L.ws);
    // which paths the policy leaves open: never dense (0), always dense (2), or either
    const bool can_dense = pol.adaptive != 0, can_pici = pol.adaptive != 2;
    // step 0: compress every rank's first chunk into slot 0 and measure sigma0;
    // ranks whose first send is dense encode it again
    SPCCL_TRY(batched_encode(L, all, kNoGate, false, m, dtype, [&](int r) { return chunk(r, (r - 1 + P) % P); },
                             [&](int r) { return L.slot(0, r, P); }, st));
    SPCCL_TRY(launch_ring_decide(ring_args(L, P, m, dtype, pol, kDecideFirst, 0), st));
    if (can_dense)
        SPCCL_TRY(batched(L, all, Gate{L.rr, -1, SPCCL_FMT_DENSE},
                          [&](int r) { return RankPtrs{chunk(r, (r - 1 + P) % P), nullptr, L.slot(0, r, P)}; },
                          [&](const RankBatch& rb, uint32_t c) { return launch_encode_dense_rb_dt(dtype, m, rb, c, st); }));
    for (int step = 1; step <= P - 1; step++) {
        SPCCL_TRY(launch_ring_decide(ring_args(L, P, m, dtype, pol, kDecideStep, step), st));
        // every send of the previous step arrives: rank r receives rank r-1's message
        SPCCL_TRY(batched(L, all, kNoGate,
                          [&](int r) { return RankPtrs{L.slot(0, (r - 1 + P) % P, P), nullptr, L.slot(1, r, P)}; },
                          [&](const RankBatch& rb, uint32_t c) {
                              return launch_copy_message_rb(L.slot_bytes, L.slot_bytes, ctrl, rb, c, st);
                          }));
        const bool last = step == P - 1;
        auto ptrs = [&](int r) {
            return RankPtrs{L.slot(1, r, P), chunk(r, (r - step - 1 + 2 * P) % P),
                            last ? static_cast<uint8_t*>(out[r]) : L.slot(0, r, P)};
        };
        for (int in_pici = 1; in_pici >= 0; in_pici--) {
            // a received message is dense only where a dense send can occur
            if (in_pici ? !can_pici : !can_dense) continue;
            const int in_fmt = in_pici ? SPCCL_FMT_PICI : SPCCL_FMT_DENSE;
            const DevOperand a_op = in_pici ? msg_op(L) : dense_msg_op(L);
            const int sa = in_pici ? SRC_PICI : SRC_DENSE;
            if (!last && can_pici) {
                const PiciSinkArgs g = sink_args(L, m, a_op, arr_op(m * s));
                SPCCL_TRY(batched(L, all, Gate{L.rr, in_fmt, SPCCL_FMT_PICI}, ptrs, [&](const RankBatch& rb, uint32_t c) {
                    return launch_to_pici_rb_dt(dtype, sa, SRC_DENSE, g, rb, c, st);
                }));
            }
            if (last || can_dense) {
                const DenseSinkArgs g = dense_args(L, m, a_op, arr_op(m * s), !last);
                const Gate gd{L.rr, in_fmt, last ? -1 : SPCCL_FMT_DENSE};
                SPCCL_TRY(batched(L, all, gd, ptrs, [&](const RankBatch& rb, uint32_t c) {
                    return launch_to_dense_rb_dt(dtype, sa, SRC_DENSE, g, rb, c, st);
                }));
            }
        }
    }
    return SPCCL_OK;
}

// All-gather of P parts of `len` elements: part q is encoded once by rank q
// (slot 0 holds those messages, of any format), travels the ring unchanged,
// and is expanded into out[r] + q*len by every rank r != q; each rank's own
// part is copied from own[r] unless it already sits in place.  One copy
// launch and one expansion launch per hop.
spccl_status_t ring_ag_batched(void* const* own, void* const* out, int P, uint64_t len, int dtype, const Layout& L,
                               hipStream_t st) {
    const uint64_t s = elem_bytes(dtype);
    for (int r = 0; r < P; r++) {
        uint8_t* dst = static_cast<uint8_t*>(out[r]) + (uint64_t)r * len * s;
        if (len && dst != own[r] && hipMemcpyAsync(dst, own[r], len * s, hipMemcpyDeviceToDevice, st) != hipSuccess)
            return SPCCL_ERR_HIP;
    }
    std::vector<int> all(P);
    for (int r = 0; r < P; r++) all[r] = r;
    WsCtrl* ctrl = reinterpret_cast<WsCtrl*>(L.ws);
    for (int k = 0; k < P - 1; k++) {
        const int in_slot = 1 + (k % 2), prev_slot = k == 0 ? 0 : 1 + ((k - 1) % 2);
        SPCCL_TRY(batched(L, all, kNoGate,
                          [&](int r) { return RankPtrs{L.slot(prev_slot, (r - 1 + P) % P, P), nullptr, L.slot(in_slot, r, P)}; },
                          [&](const RankBatch& rb, uint32_t c) {
                              return launch_copy_message_rb(L.slot_bytes, L.slot_bytes, ctrl, rb, c, st);
                          }));
        SPCCL_TRY(batched(L, all, kNoGate,
                          [&](int r) {
                              const int q = ((r - 1 - k) % P + P) % P;
                              return RankPtrs{L.slot(in_slot, r, P), nullptr,
                                              static_cast<uint8_t*>(out[r]) + (uint64_t)q * len * s};
                          },
                          [&](const RankBatch& rb, uint32_t c) {
                              return launch_gather_rb_dt(dtype, msg_op(L), len, ctrl, rb, c, st);
                          }));
    }
    return SPCCL_OK;
}

// The trace written on the device into the caller's array (entries [0, count)).
spccl_status_t copy_trace(const Layout& L, spccl_trace_t* trace, uint64_t count, hipStream_t st) {
    if (!trace || !count) return SPCCL_OK;
    return hipMemcpyAsync(trace, L.dtrace, sizeof(spccl_trace_t) * count, hipMemcpyDeviceToHost, st) == hipSuccess
               ? SPCCL_OK : SPCCL_ERR_HIP;
}

// Reduce-scatter over the chunks; the reduced chunk r goes to out[r] (m
// elements).  On return sig0 / sigp hold each rank's sigma0 and tracked
// sparsity after its last send.
spccl_status_t ring_rs(void* const* send, void* const* out, int P, uint64_t n, int dtype, const spccl_policy_t& pol,
                       const Layout& L, spccl_trace_t* trace, std::vector<double>& sig0, std::vector<double>& sigp,
                       hipStream_t st) {
    const uint64_t m = n / (uint64_t)P, s = elem_bytes(dtype);
    sig0.assign(P, 1.0);
    sigp.assign(P, 1.0);
    if (P == 1) {
        if (m && hipMemcpyAsync(out[0], send[0], m * s, hipMemcpyDeviceToDevice, st) != hipSuccess) return SPCCL_ERR_HIP;
        return SPCCL_OK;
    }
    const int sfmt = pol.sparse_fmt;
    std::vector<int> fmt(P);
    std::vector<spccl_header_t> h;
    // step 0: compress the first chunk of every rank into slot 0
    for (int r = 0; r < P; r++) {
        const int c = (r - 1 + P) % P;
        const uint8_t* chunk = static_cast<const uint8_t*>(send[r]) + (uint64_t)c * m * s;
        SPCCL_TRY(compress_fmt(sfmt, chunk, m, dtype, L, L.slot(0, r, P), st));
    }
    SPCCL_TRY(read_headers(L, 0, P, h, st));
    for (int r = 0; r < P; r++) {
        const uint64_t nnz = h[r].nnz;
        sig0[r] = sigp[r] = sparsity(m, nnz);
        fmt[r] = sfmt;
        if (send_dense(pol, sig0[r], link_tau(pol, r, P))) {
            const int c = (r - 1 + P) % P;
            const uint8_t* chunk = static_cast<const uint8_t*>(send[r]) + (uint64_t)c * m * s;
            SPCCL_TRY(spccl_encode_dense(chunk, m, dtype, L.slot(0, r, P), L.slot_bytes, st));
            fmt[r] = SPCCL_FMT_DENSE;
        }
        const uint64_t bytes = fmt[r] == sfmt ? h[r].total_bytes : dense_msg_bytes(m, dtype);
        put_trace(trace, r, 0, r, fmt[r], 1, bytes, nnz, sigp[r]);
    }
    for (int step = 1; step <= P - 1; step++) {
        // every send of the previous step arrives: rank r receives rank r-1's message
        for (int r = 0; r < P; r++)
            SPCCL_TRY(spccl_copy_message(L.slot(0, (r - 1 + P) % P, P), L.slot_bytes, L.slot(1, r, P), L.slot_bytes,
                                         L.ws, L.ws_bytes, st));
        std::vector<int> in_fmt(P);
        for (int r = 0; r < P; r++) in_fmt[r] = fmt[(r - 1 + P) % P];
        bool any_measured = false;
        for (int r = 0; r < P; r++) {
            const int c = (r - step - 1 + 2 * P) % P;
            const uint8_t* own = static_cast<const uint8_t*>(send[r]) + (uint64_t)c * m * s;
            const spccl_operand_t in = msg(L.slot(1, r, P), in_fmt[r], L.slot_bytes);
            if (step == P - 1) {   // the last receive completes chunk r
                SPCCL_TRY(spccl_reduce(in, arr(own, m * s), arr(out[r], m * s), m, dtype, L.ws, L.ws_bytes, st));
                continue;
            }
            const double est = sigp[r] * sig0[r];   // Eq. 7
            if (send_dense(pol, est, link_tau(pol, r, P))) {
                SPCCL_TRY(spccl_reduce(in, arr(own, m * s), msg(L.slot(0, r, P), SPCCL_FMT_DENSE, L.slot_bytes), m,
                                       dtype, L.ws, L.ws_bytes, st));
                fmt[r] = SPCCL_FMT_DENSE;
                sigp[r] = est;
                put_trace(trace, step * P + r, step, r, SPCCL_FMT_DENSE, 0, dense_msg_bytes(m, dtype),
                          SPCCL_NNZ_UNKNOWN, est);
            } else {
                SPCCL_TRY(spccl_reduce(in, arr(own, m * s), msg(L.slot(0, r, P), sfmt, L.slot_bytes), m, dtype,
                                       L.ws, L.ws_bytes, st));
                fmt[r] = sfmt;
                any_measured = true;
            }
        }
        if (any_measured) {
            SPCCL_TRY(read_headers(L, 0, P, h, st));
            for (int r = 0; r < P; r++) {
                if (fmt[r] != sfmt) continue;
                sigp[r] = sparsity(m, h[r].nnz);
                put_trace(trace, step * P + r, step, r, sfmt, 1, h[r].total_bytes, h[r].nnz, sigp[r]);
            }
        }
    }
    return SPCCL_OK;
}

// Pici sends over more than one rank run batched, decided on the device;
// COO sends (and a single rank) run per rank, decided on the host.
bool device_ring(const spccl_policy_t& pol, int P) { return pol.sparse_fmt == SPCCL_FMT_PICI && P > 1; }

spccl_status_t check_common(void* const* send, void* const* recv, int32_t P, int32_t dtype, void* scratch,
                            uint64_t scratch_bytes, uint64_t msg_elems) {
    if (dtype != SPCCL_F32 && dtype != SPCCL_BF16) return SPCCL_ERR_UNSUPPORTED;
    if (msg_elems >= (1ull << 32)) return SPCCL_ERR_UNSUPPORTED;
    if (!send || !recv || P < 1 || !scratch || (reinterpret_cast<uintptr_t>(scratch) & 15u))
        return SPCCL_ERR_INVALID_ARG;
    const uintptr_t amask = (uintptr_t)elem_bytes(dtype) - 1;
    for (int r = 0; r < P; r++)
        if (!send[r] || !recv[r] || (reinterpret_cast<uintptr_t>(send[r]) & amask) ||
            (reinterpret_cast<uintptr_t>(recv[r]) & amask))
            return SPCCL_ERR_INVALID_ARG;
    if (scratch_bytes < scratch_need(P, msg_elems, dtype)) return SPCCL_ERR_WORKSPACE;
    return SPCCL_OK;
}

// Which layout of a rank's receive buffer inside its own send buffer (or the
// reverse) a collective handles: the reduce-scatter writes chunk r of rank r
// last, after reading it, so recv[r] may be that chunk of send[r]; the
// all-gather reads every part before writing, so send[r] may sit at part r of
// recv[r]; the all-reduce reduces into recv while chunks are still read.
enum InPlace { kInPlaceNone, kInPlaceRsChunk, kInPlaceAgPart };

// Every overlap among the P send buffers (send_bytes each), the P receive
// buffers (recv_bytes each) and the scratch the collective uses, other than
// the one in-place layout, is rejected before anything is launched: a receive
// buffer written by one rank while another still reads it would change
// results silently.  Send buffers may overlap each other (they are only
// read).
spccl_status_t check_disjoint(void* const* send, uint64_t send_bytes, void* const* recv, uint64_t recv_bytes,
                              int32_t P, InPlace ip, uint64_t part_bytes, const void* scratch,
                              uint64_t scratch_used) {
    for (int r = 0; r < P; r++) {
        if (overlaps(recv[r], recv_bytes, scratch, scratch_used) || overlaps(send[r], send_bytes, scratch, scratch_used))
            return SPCCL_ERR_INVALID_ARG;
        for (int q = 0; q < P; q++) {
            if (q != r && overlaps(recv[r], recv_bytes, recv[q], recv_bytes)) return SPCCL_ERR_INVALID_ARG;
            if (!overlaps(recv[r], recv_bytes, send[q], send_bytes)) continue;
            const uint8_t* rb = static_cast<const uint8_t*>(recv[r]);
            const uint8_t* sb = static_cast<const uint8_t*>(send[q]);
            const bool allowed = q == r && ((ip == kInPlaceRsChunk && rb == sb + (uint64_t)r * part_bytes) ||
                                            (ip == kInPlaceAgPart && sb == rb + (uint64_t)r * part_bytes));
            if (!allowed) return SPCCL_ERR_INVALID_ARG;
        }
    }
    return SPCCL_OK;
}

spccl_status_t finish(const Layout& L, hipStream_t st) {
    return spccl_read_status(L.ws, 1, st);
}

}  // namespace

extern "C" {

uint64_t spccl_vr_scratch_bytes(int32_t P, uint64_t msg_elems, int32_t dtype) {
    if (P < 1 || (dtype != SPCCL_F32 && dtype != SPCCL_BF16)) return 0;
    return scratch_need(P, msg_elems, dtype);
}

spccl_status_t spccl_vr_reduce_scatter(void* const* send, void* const* recv, int32_t P, uint64_t n, int32_t dtype,
                                       const spccl_policy_t* policy, void* scratch, uint64_t scratch_bytes,
                                       spccl_trace_t* trace, void* stream) {
    if (P < 1 || n % (uint64_t)P) return SPCCL_ERR_INVALID_ARG;
    const uint64_t m = n / (uint64_t)P, s = elem_bytes(dtype);
    SPCCL_TRY(check_common(send, recv, P, dtype, scratch, scratch_bytes, m));
    SPCCL_TRY(check_disjoint(send, n * s, recv, m * s, P, kInPlaceRsChunk, m * s, scratch, scratch_need(P, m, dtype)));
    const spccl_policy_t pol = policy ? *policy : kDefaultPolicy;
    if (!policy_ok(pol)) return SPCCL_ERR_INVALID_ARG;
    hipStream_t st = as_stream(stream);
    const Layout L = carve(scratch, P, m, dtype);
    SPCCL_TRY(init_scratch(L, P, m, dtype, st));
    if (device_ring(pol, P)) {
        SPCCL_TRY(ring_rs_dev(send, recv, P, n, dtype, pol, L, st));
        SPCCL_TRY(copy_trace(L, trace, (uint64_t)P * (uint64_t)(P - 1), st));
    } else {
        std::vector<double> sig0, sigp;
        SPCCL_TRY(ring_rs(send, recv, P, n, dtype, pol, L, trace, sig0, sigp, st));
    }
    return finish(L, st);
}

spccl_status_t spccl_vr_all_gather(void* const* send, void* const* recv, int32_t P, uint64_t n, int32_t dtype,
                                   const spccl_policy_t* policy, void* scratch, uint64_t scratch_bytes,
                                   spccl_trace_t* trace, void* stream) {
    SPCCL_TRY(check_common(send, recv, P, dtype, scratch, scratch_bytes, n));
    const uint64_t s = elem_bytes(dtype);
    SPCCL_TRY(check_disjoint(send, n * s, recv, (uint64_t)P * n * s, P, kInPlaceAgPart, n * s, scratch,
                             scratch_need(P, n, dtype)));
    const spccl_policy_t pol = policy ? *policy : kDefaultPolicy;
    if (!policy_ok(pol)) return SPCCL_ERR_INVALID_ARG;
    hipStream_t st = as_stream(stream);
    const Layout L = carve(scratch, P, n, dtype);
    SPCCL_TRY(init_scratch(L, P, n, dtype, st));
    if (pol.sparse_fmt == SPCCL_FMT_PICI) {
        std::vector<int> all(P);
        for (int q = 0; q < P; q++) all[q] = q;
        SPCCL_TRY(batched_encode(L, all, kNoGate, false, n, dtype,
                                 [&](int q) { return static_cast<const uint8_t*>(send[q]); },
                                 [&](int q) { return L.slot(0, q, P); }, st));
        SPCCL_TRY(launch_ring_decide(ring_args(L, P, n, dtype, pol, kDecideAllGather, 0), st));
        SPCCL_TRY(copy_trace(L, trace, (uint64_t)P, st));
    } else {
        for (int q = 0; q < P; q++) SPCCL_TRY(compress_fmt(pol.sparse_fmt, send[q], n, dtype, L, L.slot(0, q, P), st));
        std::vector<spccl_header_t> h;
        SPCCL_TRY(read_headers(L, 0, P, h, st));
        for (int q = 0; q < P; q++)
            put_trace(trace, q, 0, q, pol.sparse_fmt, 1, h[q].total_bytes, h[q].nnz, sparsity(n, h[q].nnz));
    }
    SPCCL_TRY(ring_ag_batched(send, recv, P, n, dtype, L, st));
    return finish(L, st);
}

spccl_status_t spccl_vr_all_reduce(void* const* send, void* const* recv, int32_t P, uint64_t n, int32_t dtype,
                                   const spccl_policy_t* policy, void* scratch, uint64_t scratch_bytes,
                                   spccl_trace_t* trace, void* stream) {
    if (P < 1 || n % (uint64_t)P) return SPCCL_ERR_INVALID_ARG;
    const uint64_t m = n / (uint64_t)P, s = elem_bytes(dtype);
    SPCCL_TRY(check_common(send, recv, P, dtype, scratch, scratch_bytes, m));
    // outputs must not overlap the inputs (chunks are reduced into them), each other or the scratch
    SPCCL_TRY(check_disjoint(send, n * s, recv, n * s, P, kInPlaceNone, 0, scratch, scratch_need(P, m, dtype)));
    const spccl_policy_t pol = policy ? *policy : kDefaultPolicy;
    if (!policy_ok(pol)) return SPCCL_ERR_INVALID_ARG;
    hipStream_t st = as_stream(stream);
    const Layout L = carve(scratch, P, m, dtype);
    SPCCL_TRY(init_scratch(L, P, m, dtype, st));
    // reduce-scatter straight into each rank's own chunk of its output
    std::vector<void*> chunk_out(P);
    for (int r = 0; r < P; r++) chunk_out[r] = static_cast<uint8_t*>(recv[r]) + (uint64_t)r * m * s;
    if (device_ring(pol, P)) {
        // the transition decided on the device from each rank's tracked sparsity
        std::vector<int> all(P);
        for (int r = 0; r < P; r++) all[r] = r;
        SPCCL_TRY(ring_rs_dev(send, chunk_out.data(), P, n, dtype, pol, L, st));
        SPCCL_TRY(launch_ring_decide(ring_args(L, P, m, dtype, pol, kDecideGather, 0), st));
        SPCCL_TRY(batched_encode(L, all, Gate{L.rr, -1, -1}, pol.adaptive != 0, m, dtype,
                                 [&](int r) { return static_cast<const uint8_t*>(chunk_out[r]); },
                                 [&](int r) { return L.slot(0, r, P); }, st));
        SPCCL_TRY(launch_ring_decide(ring_args(L, P, m, dtype, pol, kDecideGatherSizes, 0), st));
        SPCCL_TRY(copy_trace(L, trace, (uint64_t)P * (uint64_t)(P - 1) + (uint64_t)P, st));
    } else {
        std::vector<double> sig0, sigp;
        SPCCL_TRY(ring_rs(send, chunk_out.data(), P, n, dtype, pol, L, trace, sig0, sigp, st));
        // phase-aware transition: one message per rank, encoded once
        std::vector<int> fmt(P);
        std::vector<double> est(P);
        for (int r = 0; r < P; r++) {
            est[r] = sigp[r] * sig0[r];
            const bool dense = pol.adaptive == 2 ? true : (pol.adaptive == 0 ? false : est[r] <= pol.ag_thresh);
            fmt[r] = dense ? SPCCL_FMT_DENSE : pol.sparse_fmt;
            if (dense) SPCCL_TRY(spccl_encode_dense(chunk_out[r], m, dtype, L.slot(0, r, P), L.slot_bytes, stream));
            else SPCCL_TRY(compress_fmt(pol.sparse_fmt, chunk_out[r], m, dtype, L, L.slot(0, r, P), st));
        }
        std::vector<spccl_header_t> h;
        SPCCL_TRY(read_headers(L, 0, P, h, st));
        spccl_trace_t* ag_tr = trace ? trace + (uint64_t)P * (uint64_t)(P - 1) : nullptr;
        for (int r = 0; r < P; r++) {
            const bool sparse = fmt[r] != SPCCL_FMT_DENSE;
            put_trace(ag_tr, r, P - 1, r, fmt[r], sparse ? 1 : 0, h[r].total_bytes,
                      sparse ? h[r].nnz : SPCCL_NNZ_UNKNOWN, est[r]);
        }
    }
    SPCCL_TRY(ring_ag_batched(chunk_out.data(), recv, P, m, dtype, L, st));
    return finish(L, st);
}

/* ---- sliced ring collectives: decisions on the device ------------------------ */

namespace {
struct SlicedLayout {
    uint8_t* ws;           // control block
    double* track;         // P trackers of S slices
    uint8_t* fmt;          // (P-1) * P * S reduce-scatter formats, then P * S all-gather formats
    uint8_t* streams;      // 2 * P sliced streams (sent, received)
    uint64_t S, sbytes, track_bytes;
    uint8_t* stream(int which, int r, int P) const { return streams + ((uint64_t)which * P + r) * sbytes; }
};

uint64_t sliced_need(int32_t P, uint64_t m, int32_t dtype, SlicedLayout* L, void* base) {
    const uint64_t S = spccl_slice_count(m);
    const uint64_t sbytes = round_up(S * spccl_slice_bytes(dtype));
    const uint64_t wsb = round_up(kWsFlagsOffset), trb = round_up(16ull * S * (uint64_t)P),
                   fmb = round_up((uint64_t)P * (uint64_t)P * S);    // reduce-scatter steps, then an all-gather
    if (L) {
        uint8_t* b = static_cast<uint8_t*>(base);
        L->ws = b;
        L->track = reinterpret_cast<double*>(b + wsb);
        L->fmt = b + wsb + trb;
        L->streams = b + wsb + trb + fmb;
        L->S = S;
        L->sbytes = sbytes;
        L->track_bytes = 16ull * S;
    }
    return wsb + trb + fmb + 2ull * (uint64_t)P * sbytes;
}

// The policy as one threshold per link: adaptive 0 never goes dense (no
// sparsity is below -1), adaptive 2 always does (none is above 2).
double sliced_tau(const spccl_policy_t& pol, int r, int P) {
    if (pol.adaptive == 0) return -1.0;
    if (pol.adaptive == 2) return 2.0;
    return link_tau(pol, r, P);
}
}  // namespace

uint64_t spccl_vr_sliced_scratch_bytes(int32_t P, uint64_t msg_elems, int32_t dtype) {
    if (P < 1 || (dtype != SPCCL_F32 && dtype != SPCCL_BF16)) return 0;
    return sliced_need(P, msg_elems, dtype, nullptr, nullptr);
}

namespace {

// Buffers of the sliced collectives: P send buffers of send_elems and P
// receive buffers of recv_elems elements, element-aligned; no receive
// buffer may overlap another or any send buffer, because the ranks of a step
// share one launch.
spccl_status_t check_sliced_ranks(void* const* send, uint64_t send_elems, void* const* recv, uint64_t recv_elems,
                                  int32_t P, int32_t dtype, const void* scratch, uint64_t scratch_used) {
    const uint64_t s = elem_bytes(dtype);
    if (!send || !recv || !scratch || (reinterpret_cast<uintptr_t>(scratch) & 15u)) return SPCCL_ERR_INVALID_ARG;
    const uintptr_t amask = (uintptr_t)s - 1;
    for (int r = 0; r < P; r++)
        if (!send[r] || !recv[r] || (reinterpret_cast<uintptr_t>(send[r]) & amask) ||
            (reinterpret_cast<uintptr_t>(recv[r]) & amask))
            return SPCCL_ERR_INVALID_ARG;
    for (int r = 0; r < P; r++) {
        if (overlaps(recv[r], recv_elems * s, scratch, scratch_used) ||
            overlaps(send[r], send_elems * s, scratch, scratch_used))
            return SPCCL_ERR_INVALID_ARG;
        for (int q = 0; q < P; q++)
            if (overlaps(recv[r], recv_elems * s, send[q], send_elems * s) ||
                (q != r && overlaps(recv[r], recv_elems * s, recv[q], recv_elems * s)))
                return SPCCL_ERR_INVALID_ARG;
    }
    return SPCCL_OK;
}

SlicedBatch make_batch(const SlicedLayout& L, uint64_t m, int32_t dtype, uint8_t* out0, const uint8_t* b0,
                       double* track0, int32_t track_step, uint8_t* fmt0) {
    SlicedBatch b{};
    b.base = SlicedArgs{nullptr, b0, out0, m, slice_slot_bytes(dtype), 0.0, reinterpret_cast<WsCtrl*>(L.ws), track0,
                        track_step, fmt0};
    b.b_stride = L.sbytes;
    b.out_stride = L.sbytes;
    b.track_stride = 2 * L.S;
    b.fmt_stride = L.S;
    return b;
}

inline int batch_count(int P, int r0) { return P - r0 < kMaxBatchRanks ? P - r0 : kMaxBatchRanks; }

// The sliced reduce-scatter's steps (m > 0, P > 1): every step is one launch
// per kernel for up to kMaxBatchRanks ranks (grid y = rank), the P
// reductions of a ring step being independent; rank r's reduced chunk lands
// at out[r].  Formats go to L.fmt, step-major.
spccl_status_t sliced_rs_steps(void* const* send, uint8_t* const* out, int32_t P, uint64_t m, int32_t dtype,
                               const spccl_policy_t& pol, const SlicedLayout& L, hipStream_t st) {
    const uint64_t s = elem_bytes(dtype);
    auto chunk = [&](int r, int c) { return static_cast<const uint8_t*>(send[r]) + (uint64_t)c * m * s; };
    auto fmt_at = [&](int step, int r) { return L.fmt + ((uint64_t)step * P + r) * L.S; };
    for (int step = 0; step <= P - 1; step++) {
        if (step > 0)   // the sends: rank r receives rank r-1's stream
            for (int r0 = 0; r0 < P; r0 += kMaxBatchRanks) {
                SlicedBatch c = make_batch(L, m, dtype, L.stream(1, r0, P), nullptr, nullptr, 0, nullptr);
                for (int j = 0; j < batch_count(P, r0); j++) c.a[j] = L.stream(0, (r0 + j - 1 + P) % P, P);
                SPCCL_TRY(launch_copy_sliced_batch(c, (uint32_t)batch_count(P, r0), st));
            }
        for (int r0 = 0; r0 < P; r0 += kMaxBatchRanks) {
            const int cnt = batch_count(P, r0);
            const bool first = step == 0, last = step == P - 1;
            // step 0 compresses each rank's first chunk and starts its slices'
            // trackers; later steps reduce the received stream into the own
            // chunk (Eq. 7 per slice); the last one into the dense output
            SlicedBatch b = last ? make_batch(L, m, dtype, nullptr, L.stream(1, r0, P), nullptr, 0, nullptr)
                                 : make_batch(L, m, dtype, L.stream(0, r0, P), first ? nullptr : L.stream(1, r0, P),
                                              L.track + 2 * L.S * r0, first ? 0 : 1, fmt_at(step, r0));
            for (int j = 0; j < cnt; j++) {
                const int r = r0 + j;
                b.a[j] = chunk(r, (r - step - 1 + 2 * P) % P);
                b.thresh[j] = last ? 0.0 : sliced_tau(pol, r, P);
                if (last) b.out_dense[j] = out[r];
            }
            SPCCL_TRY(launch_sliced_batch_dt(dtype, b, (uint32_t)cnt,
                                             first ? kSlicedCompress : (last ? kSlicedReduceToDense : kSlicedReduceToSliced),
                                             st));
        }
    }
    return SPCCL_OK;
}

// The sliced all-gather's hops (n_part > 0): stream(0, r) holds rank r's
// encoded part; rank r expands it into its own place (unless own_in_place:
// the part is already there), then at hop k receives rank r-k's stream into
// stream(1, r) and expands it into part r-k of recv[r].  One launch per
// kernel and hop for up to kMaxBatchRanks ranks.
spccl_status_t sliced_ag_hops(void* const* recv, int32_t P, uint64_t n_part, int32_t dtype, const SlicedLayout& L,
                              bool own_in_place, hipStream_t st) {
    const uint64_t s = elem_bytes(dtype);
    auto place = [&](int r, int q) { return static_cast<uint8_t*>(recv[r]) + (uint64_t)q * n_part * s; };
    for (int k = own_in_place ? 1 : 0; k <= P - 1; k++) {
        for (int r0 = 0; r0 < P; r0 += kMaxBatchRanks) {
            const int cnt = batch_count(P, r0);
            if (k > 0) {
                SlicedBatch c = make_batch(L, n_part, dtype, L.stream(1, r0, P), nullptr, nullptr, 0, nullptr);
                for (int j = 0; j < cnt; j++) c.a[j] = L.stream(0, (r0 + j - k + P) % P, P);
                SPCCL_TRY(launch_copy_sliced_batch(c, (uint32_t)cnt, st));
            }
            SlicedBatch e = make_batch(L, n_part, dtype, nullptr, nullptr, nullptr, 0, nullptr);
            for (int j = 0; j < cnt; j++) {
                const int r = r0 + j;
                e.a[j] = k == 0 ? L.stream(0, r, P) : L.stream(1, r, P);
                e.out_dense[j] = place(r, (r - k + P) % P);
            }
            SPCCL_TRY(launch_sliced_batch_dt(dtype, e, (uint32_t)cnt, kSlicedExpand, st));
        }
    }
    return SPCCL_OK;
}

spccl_status_t copy_to_host(void* dst, const void* src, uint64_t bytes, hipStream_t st) {
    if (!dst || !bytes) return SPCCL_OK;
    return hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, st) == hipSuccess ? SPCCL_OK : SPCCL_ERR_HIP;
}

}  // namespace

spccl_status_t spccl_vr_reduce_scatter_sliced(void* const* send, void* const* recv, int32_t P, uint64_t n,
                                              int32_t dtype, const spccl_policy_t* policy, void* scratch,
                                              uint64_t scratch_bytes, uint8_t* fmt_trace, void* stream) {
    if (P < 1 || n % (uint64_t)P) return SPCCL_ERR_INVALID_ARG;
    const uint64_t m = n / (uint64_t)P, s = elem_bytes(dtype);
    if (dtype != SPCCL_F32 && dtype != SPCCL_BF16) return SPCCL_ERR_UNSUPPORTED;
    if (m >= (1ull << 32)) return SPCCL_ERR_UNSUPPORTED;
    SPCCL_TRY(check_sliced_ranks(send, n, recv, m, P, dtype, scratch, sliced_need(P, m, dtype, nullptr, nullptr)));
    const spccl_policy_t pol = policy ? *policy : kDefaultPolicy;
    if (!policy_ok(pol)) return SPCCL_ERR_INVALID_ARG;
    if (pol.sparse_fmt != SPCCL_FMT_PICI) return SPCCL_ERR_UNSUPPORTED;      // slices are Pici or dense
    if (scratch_bytes < sliced_need(P, m, dtype, nullptr, nullptr)) return SPCCL_ERR_WORKSPACE;
    hipStream_t st = as_stream(stream);
    if (P == 1) {
        if (m && hipMemcpyAsync(recv[0], send[0], m * s, hipMemcpyDeviceToDevice, st) != hipSuccess) return SPCCL_ERR_HIP;
        return hipStreamSynchronize(st) == hipSuccess ? SPCCL_OK : SPCCL_ERR_HIP;
    }
    SlicedLayout L;
    sliced_need(P, m, dtype, &L, scratch);
    SPCCL_TRY(spccl_workspace_init(L.ws, kWsFlagsOffset, stream));
    if (m == 0) return spccl_read_status(L.ws, 1, st);
    SPCCL_TRY(sliced_rs_steps(send, reinterpret_cast<uint8_t* const*>(recv), P, m, dtype, pol, L, st));
    SPCCL_TRY(copy_to_host(fmt_trace, L.fmt, (uint64_t)(P - 1) * P * L.S, st));
    return spccl_read_status(L.ws, 1, st);
}

spccl_status_t spccl_vr_all_gather_sliced(void* const* send, void* const* recv, int32_t P, uint64_t n, int32_t dtype,
                                          void* scratch, uint64_t scratch_bytes, uint8_t* fmt_trace, void* stream) {
    if (P < 1) return SPCCL_ERR_INVALID_ARG;
    if (dtype != SPCCL_F32 && dtype != SPCCL_BF16) return SPCCL_ERR_UNSUPPORTED;
    if (n >= (1ull << 32)) return SPCCL_ERR_UNSUPPORTED;
    const uint64_t s = elem_bytes(dtype);
    SPCCL_TRY(check_sliced_ranks(send, n, recv, (uint64_t)P * n, P, dtype, scratch,
                                 sliced_need(P, n, dtype, nullptr, nullptr)));
    if (scratch_bytes < sliced_need(P, n, dtype, nullptr, nullptr)) return SPCCL_ERR_WORKSPACE;
    hipStream_t st = as_stream(stream);
    if (P == 1) {
        if (n && hipMemcpyAsync(recv[0], send[0], n * s, hipMemcpyDeviceToDevice, st) != hipSuccess) return SPCCL_ERR_HIP;
        return hipStreamSynchronize(st) == hipSuccess ? SPCCL_OK : SPCCL_ERR_HIP;
    }
    SlicedLayout L;
    sliced_need(P, n, dtype, &L, scratch);
    SPCCL_TRY(spccl_workspace_init(L.ws, kWsFlagsOffset, stream));
    if (n == 0) return spccl_read_status(L.ws, 1, st);
    // every rank encodes its part once, every slice Pici (a standalone
    // all-gather does not densify)
    for (int r0 = 0; r0 < P; r0 += kMaxBatchRanks) {
        SlicedBatch b = make_batch(L, n, dtype, L.stream(0, r0, P), nullptr, nullptr, 0, L.fmt + (uint64_t)r0 * L.S);
        for (int j = 0; j < batch_count(P, r0); j++) {
            b.a[j] = static_cast<const uint8_t*>(send[r0 + j]);
            b.thresh[j] = -1.0;
        }
        SPCCL_TRY(launch_sliced_batch_dt(dtype, b, (uint32_t)batch_count(P, r0), kSlicedCompress, st));
    }
    SPCCL_TRY(sliced_ag_hops(recv, P, n, dtype, L, false, st));
    SPCCL_TRY(copy_to_host(fmt_trace, L.fmt, (uint64_t)P * L.S, st));
    return spccl_read_status(L.ws, 1, st);
}

spccl_status_t spccl_vr_all_reduce_sliced(void* const* send, void* const* recv, int32_t P, uint64_t n, int32_t dtype,
                                          const spccl_policy_t* policy, void* scratch, uint64_t scratch_bytes,
                                          uint8_t* fmt_rs, uint8_t* fmt_ag, void* stream) {
    if (P < 1 || n % (uint64_t)P) return SPCCL_ERR_INVALID_ARG;
    const uint64_t m = n / (uint64_t)P, s = elem_bytes(dtype);
    if (dtype != SPCCL_F32 && dtype != SPCCL_BF16) return SPCCL_ERR_UNSUPPORTED;
    if (m >= (1ull << 32)) return SPCCL_ERR_UNSUPPORTED;
    SPCCL_TRY(check_sliced_ranks(send, n, recv, n, P, dtype, scratch, sliced_need(P, m, dtype, nullptr, nullptr)));
    const spccl_policy_t pol = policy ? *policy : kDefaultPolicy;
    if (!policy_ok(pol)) return SPCCL_ERR_INVALID_ARG;
    if (pol.sparse_fmt != SPCCL_FMT_PICI) return SPCCL_ERR_UNSUPPORTED;
    if (scratch_bytes < sliced_need(P, m, dtype, nullptr, nullptr)) return SPCCL_ERR_WORKSPACE;
    hipStream_t st = as_stream(stream);
    if (P == 1) {
        if (n && hipMemcpyAsync(recv[0], send[0], n * s, hipMemcpyDeviceToDevice, st) != hipSuccess) return SPCCL_ERR_HIP;
        return hipStreamSynchronize(st) == hipSuccess ? SPCCL_OK : SPCCL_ERR_HIP;
    }
    SlicedLayout L;
    sliced_need(P, m, dtype, &L, scratch);
    SPCCL_TRY(spccl_workspace_init(L.ws, kWsFlagsOffset, stream));
    if (m == 0) return spccl_read_status(L.ws, 1, st);
    // reduce-scatter: rank r's reduced chunk lands in its own place in recv[r]
    std::vector<uint8_t*> own(P);
    for (int r = 0; r < P; r++) own[r] = static_cast<uint8_t*>(recv[r]) + (uint64_t)r * m * s;
    SPCCL_TRY(sliced_rs_steps(send, own.data(), P, m, dtype, pol, L, st));
    // transition (Sec. IV-C per slice): est = sigma_prev * sigma0 from the
    // slice's tracker; the slice is gathered densely iff est <= ag_thresh
    const double ag_tau = pol.adaptive == 0 ? -1.0 : (pol.adaptive == 2 ? 2.0 : pol.ag_thresh);
    uint8_t* fmt_ag_dev = L.fmt + (uint64_t)(P - 1) * P * L.S;
    for (int r0 = 0; r0 < P; r0 += kMaxBatchRanks) {
        SlicedBatch b = make_batch(L, m, dtype, L.stream(0, r0, P), nullptr, L.track + 2 * L.S * r0, 1,
                                   fmt_ag_dev + (uint64_t)r0 * L.S);
        for (int j = 0; j < batch_count(P, r0); j++) {
            b.a[j] = own[r0 + j];
            b.thresh[j] = ag_tau;
        }
        SPCCL_TRY(launch_sliced_batch_dt(dtype, b, (uint32_t)batch_count(P, r0), kSlicedCompress, st));
    }
    SPCCL_TRY(sliced_ag_hops(recv, P, m, dtype, L, true, st));
    SPCCL_TRY(copy_to_host(fmt_rs, L.fmt, (uint64_t)(P - 1) * P * L.S, st));
    SPCCL_TRY(copy_to_host(fmt_ag, fmt_ag_dev, (uint64_t)P * L.S, st));
    return spccl_read_status(L.ws, 1, st);
}

}  // extern "C"

