// resispec.hip -- gfx950 kernels and C ABI of the ResiSpec verification step.
//
// Paper: "ResiSpec: Enhancing Multi-Candidate Speculative Sampling via Residual
// Distribution Shaping".  One workgroup verifies one tree node (one logits row):
//
//   pass 1   softmax statistics (sums of exp) of the target row and, for nodes with
//            children, the draft row (Preliminary; temperature T);
//   tests    candidate i is accepted iff u_i < R_i(x_i) / D_i(x_i) (Eq. 2 and
//            Algorithm 1), evaluated in fp64 on the gathered candidate logits;
//   pass i+1 after the i-th rejection one more pass over the row computes the sums the
//            residual update needs:
//              standard (Eq. 1/2):   Tot = sum_j max(p_j - C_i q_j, 0); applying
//                                    max(R - D, 0) / S i times gives
//                                    max(p - C_i q, 0) / Tot with C_i from the earlier
//                                    totals, so one step per element for any i;
//              ResiSpec (Algorithm 1, GetProxy): M = sum_{j != x0} min(Z D_j, R_j), with
//                                    Z = D(x0) - R(x0); SR = sum_{j != x0} R_j is
//                                    1 - R(x0) because R is normalised.
//            GetProxy's one-shot redistribution of Delta = Z - M into the capacity
//            R_j - m_j gives, with a = Delta / (SR - M), the residual
//              R'_j = ((1 - a) min(Z D_j, R_j) + a R_j) / Z   (j != x0),   R'_x0 = 0,
//            i.e. norm(max(R - K, 0)) for the proxy K = R - r, K(x0) = D(x0).  So the
//            residual is never materialised: every pass re-derives R_j from the two
//            logits of token j through the chain of per-rejection scalars.  After the
//            first rejection pass min(c Q, R) = exp2(min(log2 R, log2 Q + log2 c))
//            takes a single exponential per element, and each later step of the chain
//            is min(a/Z R + (1 - a) c/Z Q, R/Z);
//   draw     when every candidate is rejected (or the node is a leaf: bonus draw from
//            p), the token is the smallest j whose running sum of the final residual in
//            vocabulary order exceeds u * total.  The last pass records partial sums
//            per slot (a run of G chunks of 64 * VEC * UNR elements), so the draw
//            re-reads one slot.
//
// Numerics: elements in fp32 (bf16 widened exactly), sums of fp32 lane partials in
// fp64, the candidates' probabilities and the scalar chain in fp64.  Exponents are
// exp2(l * c2 + K) with c2 = log2(e)/T split into two floats and K an integer-valued
// reference fixed per row before pass 1 (from the first chunks' maximum; a row whose
// sums overflow or underflow against it takes an exact-maximum pass), so an element's
// value does not depend on which wave read it and every reduction runs in a fixed
// order: results are bitwise reproducible.  Residual elements are carried in units of
// the target row's unnormalised mass (the target normaliser is folded into the step
// constants).
//
// A second kernel walks each tree from the root along accepted children; a third
// (the path-only schedule) verifies only the nodes each walk reaches, and a fourth
// verifies each row of a small batch with several workgroups (row groups).  The draft
// step that precedes verification is in draft.hip; shared helpers are in common.h.

#include <atomic>
#include <mutex>

#include "common.h"

namespace {

struct KParams {
    const void* tgt;
    const void* dft;
    // flat rows
    const int32_t* cand_ids;
    const float* ua_flat;
    const float* ur_flat;
    int32_t k;
    int32_t* out_token;
    int32_t* out_len;
    int32_t* out_status;
    // tree rows
    const int32_t* node_token;
    const int32_t* parent;
    const float* ua;
    const float* ur;
    int32_t* node_child;
    int32_t* node_tok;
    int32_t* node_status;
    float* residual_out;
    // path schedule with a workspace: per-sequence fp32 residual of the running row
    // (rc_stride floats per sequence), or null
    // deferred draws (the other schedules): per node row, the pass-1 slot totals of the
    // target row, then of the draft row (kStateDoubles doubles a row), kept for the rows
    // whose draw is left to the walk
    union {
        float* rcache;
        double* dstate;
    };
    int64_t rc_stride;
    int32_t B, N;
    int32_t V;
    float T;
    float c2h, c2l;      // log2(e) / T = c2h + c2l
    int32_t worep, bonus, flat;
    int32_t G;           // chunks per slot
    int32_t nslots;      // slots per row
};


__device__ __forceinline__ void write_outcome(const KParams& P, int64_t row, int32_t child,
                                              int32_t tok, int32_t status) {
    if (P.flat) {
        const bool ok = status == RS_SEQ_OK;
        P.out_token[row] = ok ? tok : -1;
        P.out_len[row] = ok ? (child >= 0 ? 1 : 0) : -1;
        if (P.out_status) P.out_status[row] = status;
    } else {
        P.node_child[row] = status == RS_SEQ_OK ? child : -1;
        P.node_tok[row] = status == RS_SEQ_OK ? tok : -1;
        P.node_status[row] = status;
    }
}

__device__ void zero_residual_row(const KParams& P, int64_t row) {
    if (!P.residual_out) return;
    float* out = P.residual_out + row * P.V;
    for (int j = threadIdx.x; j < P.V; j += blockDim.x) out[j] = 0.0f;
}

// Rejection-step terms of one element (exact token comparisons), given its target
// mass R (target units) and unnormalised draft mass Q:
//   standard: A = max(R - C_i Q, 0)          (the collapsed recurrence, C_i = st_c[i])
//   ResiSpec: A = min(c_i Q, R), B = R, both 0 at x_i   (c_i = Z_i dscale_i St/Sd),
//             after the chain over the earlier steps 0..i-1.  A step of the chain,
//             R <- (a (R - m) + m) / Z with m = min(c Q, R), equals
//             min(a/Z R + (1 - a) c/Z Q, R/Z) because 0 <= a <= 1: four operations.
template <int MODE>
__device__ __forceinline__ void chain_terms(float R, float Q, int j, const Smem& sm, int i,
                                            float& A, float& Bv) {
    if (MODE == RS_MODE_SPECINFER) {
        A = fmaxf(fmaf(-sm.st_c[i], Q, R), 0.0f);
        Bv = 0.0f;
        return;
    }
    for (int t = 0; t < i; ++t) {
        R = fminf(fmaf(sm.st_kc[t], Q, sm.st_k1[t] * R), sm.st_i[t] * R);
        if (j == sm.st_x[t]) R = 0.0f;
    }
    const bool x0 = j == sm.st_x[i];
    A = x0 ? 0.0f : fminf(sm.st_c[i] * Q, R);
    Bv = x0 ? 0.0f : R;
}

// Scalar chain for the accept test of candidate i (fp64, normalised units): R(x) and
// D(x) of the candidate.  Returned by value (a call, if the compiler keeps one, passes
// them in registers rather than through a stack slot).
struct ResDraft {
    double R, D;
};
template <int MODE>
__device__ ResDraft scalar_residual(const Smem& sm, int i, double p, double q, int32_t x, bool worep) {
    bool removed = false;
    if (worep)
        for (int t = 0; t < i; ++t) removed |= x == sm.st_x[t];
    const double Dout = removed ? 0.0 : q * sm.st_ds[i];
    if (MODE == RS_MODE_SPECINFER) {
        // the standard recurrence max(R - D, 0) / S applied i times equals
        // max(p - C q, 0) / Tot (every factor is positive)
        if (i == 0) return {p, Dout};
        const double w = p - sm.st_C[i - 1] * q;
        return {w > 0.0 ? w / sm.st_tot[i - 1] : 0.0, Dout};
    }
    double R = p;
    removed = false;
    for (int t = 0; t < i; ++t) {
        const double Dt = removed ? 0.0 : q * sm.st_ds[t];
        if (x == sm.st_x[t]) {
            R = 0.0;
        } else {
            const double zd = sm.st_zd[t] * Dt;
            const double m = zd < R ? zd : R;
            R = ((1.0 - sm.st_ad[t]) * m + sm.st_ad[t] * R) / sm.st_zd[t];
        }
        if (worep && x == sm.st_x[t]) removed = true;
    }
    return {R, Dout};
}

// ------------------------------------------------------------ row kernel ----

// Verification of one node row by the whole workgroup: node n of sequence b (row
// b * N + n; flat rows: b = row, n = 0).  emit(child, token, status) is called by
// thread 0 once, with the node's outcome.
// Workgroups that verify one row together (row groups of the path schedule or of the
// all-nodes schedule, one workgroup per CU): member w of S sweeps slots [w * nslots / S, (w + 1) * nslots / S)
// in every pass; after a pass the members exchange their slots' totals through global
// memory, then all continue from the same totals in the same order, so each decision is
// taken identically by every member.  S = 1: one workgroup per row.
//
// The exchange needs no fence: every value travels in 64-bit atomic words that carry the
// exchange's number (the same count in every member) in their upper half and 32 bits of
// the value in the lower half, and a reader waits until each word it needs carries the
// current number.  Per-location coherence of the atomics is all this relies on, and a
// member writes exchange e + 2 into the buffer of exchange e only after reading every
// member's exchange e + 1, which each wrote after reading exchange e: two buffers are
// enough.
struct RowGroup {
    int32_t S, w;              // members, this member
    unsigned long long* xw;    // [2 (parity)][2 (first, second sum)][kMaxSlots][2 (halves)]
    unsigned long long* xm;    // [2 (parity)][kMaxGroup][2]: the members' maxima of both rows
    uint32_t epoch;            // exchanges so far (the same count in every member)
    uint64_t wait;             // time limit of one exchange, in ticks of the 100 MHz wall clock
};

// per-sequence (or per-row) workspace of a row group: formation arrivals and state (each
// on its own 64-byte line), slot totals, maxima (tagged words, zero before the launch)
constexpr int32_t kMaxGroup = 16;
constexpr int64_t kGroupArrive = 64;
constexpr int64_t kGroupState = 128;
constexpr int64_t kGroupXw = 256;
constexpr int64_t kGroupXm = kGroupXw + 2 * 2 * kMaxSlots * 2 * (int64_t)sizeof(unsigned long long);
constexpr int64_t kGroupWordsEnd = kGroupXm + 2 * kMaxGroup * 2 * (int64_t)sizeof(unsigned long long);
constexpr int64_t kGroupStride = (kGroupWordsEnd + 255) / 256 * 256;
constexpr int32_t kAutoRowGroup = 8;       // automatic members per row, all-nodes schedule, at most,
constexpr int64_t kAutoRowBytes = 40960;   // at least this many bytes of a row's logits each,
constexpr int64_t kAutoSplitBytes = 163840;   // for rows of at least this many bytes of logits
// XCDs of the device, and when groups are placed on one XCD each: groups of at most 8
// members, at least two groups per XCD (measured: a group that ends up alone on its XCD,
// of 7 or of 15, is slower confined to that XCD's share of the chip)
constexpr int64_t kXcds = 8;
constexpr int32_t kXcdMaxMembers = 8;
constexpr int64_t kXcdMinGroups = 2 * kXcds;

// Time limit of one exchange (20 ms of the 100 MHz wall clock unless a test sets
// another): a member whose partners have not published in time gives up, so every
// workgroup ends whatever happens to the others (the row then reports
// RS_SEQ_GROUP_TIMEOUT).
constexpr uint64_t kGroupWaitTicks = 2000000ull;

__device__ __forceinline__ void put_tagged(unsigned long long* w, uint32_t tag, uint32_t v) {
    __hip_atomic_store(w, ((unsigned long long)tag << 32) | v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The values of words w[0..N) once every one of them carries `tag`; false if they do not
// within `limit` ticks of t0.  All N loads are in flight together on every poll.
template <int N>
__device__ __forceinline__ bool get_tagged_all(const unsigned long long* const (&w)[N], uint32_t tag,
                                               uint32_t (&v)[N], uint64_t t0, uint64_t limit) {
    for (;;) {
        unsigned long long x[N];
#pragma unroll
        for (int k = 0; k < N; ++k) x[k] = __hip_atomic_load(w[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        bool all = true;
#pragma unroll
        for (int k = 0; k < N; ++k) all = all && (uint32_t)(x[k] >> 32) == tag;
        if (all) {
#pragma unroll
            for (int k = 0; k < N; ++k) v[k] = (uint32_t)x[k];
            return true;
        }
        if ((uint64_t)wall_clock64() - t0 > limit) return false;
        __builtin_amdgcn_s_sleep(1);
    }
}

__device__ __forceinline__ double join_halves(uint32_t lo, uint32_t hi) {
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

__device__ __forceinline__ void put_tagged_d(unsigned long long* w, uint32_t tag, double v) {
    const unsigned long long bits = (unsigned long long)__double_as_longlong(v);
    put_tagged(w, tag, (uint32_t)bits);
    put_tagged(w + 1, tag, (uint32_t)(bits >> 32));
}


// Group formation, before a group's first row.  Members are launched as ordinary
// workgroups, so they need not all be resident at once: each counts its arrival, and
// the last to arrive marks the group formed.  A member that sees no such mark within
// the formation limit (20 us unless a test sets another) claims the group's work for
// itself, and members that find it claimed leave.  The state moves once, from open to
// formed or claimed: when formed, every member is running and takes part in every exchange.
// Returns 1 (formed: work as member w of S), 2 (claimed: do all of it alone) or 0
// (leave).
constexpr uint32_t kFormOpen = 0u, kFormed = 1u, kFormClaimed = 2u;
constexpr uint64_t kFormWaitTicks = 2000ull;

__device__ __forceinline__ int form_group(Smem& sm, const RowGroup& g, char* base, uint64_t wait) {
    if (threadIdx.x == 0) {
        uint32_t* arrive = reinterpret_cast<uint32_t*>(base + kGroupArrive);
        uint32_t* state = reinterpret_cast<uint32_t*>(base + kGroupState);
        if (atomicAdd(arrive, 1u) + 1u == (uint32_t)g.S) atomicCAS(state, kFormOpen, kFormed);
        const uint64_t t0 = (uint64_t)wall_clock64();
        int res;
        for (;;) {
            const uint32_t st = __hip_atomic_load(state, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (st != kFormOpen) {
                res = st == kFormed ? 1 : 0;
                break;
            }
            if ((uint64_t)wall_clock64() - t0 > wait) {
                const uint32_t old = atomicCAS(state, kFormOpen, kFormClaimed);
                res = old == kFormOpen ? 2 : (old == kFormed ? 1 : 0);
                break;
            }
            __builtin_amdgcn_s_sleep(2);
        }
        __threadfence();
        sm.group_ok = res;
    }
    __syncthreads();
    const int res = __builtin_amdgcn_readfirstlane(sm.group_ok);
    __syncthreads();   // every thread has read group_ok
    return res;
}

// Slot totals of the pass just swept (this workgroup's slots [s0, s0 + nl)): summed in
// shared memory, then, in a row group, published and gathered, so that on return
// slotA / slotB (and slotP if keepP) hold the totals of every slot of the row.
// False if the exchange timed out.
template <int BLK, bool SPLIT>
__device__ __forceinline__ bool pass_totals(Smem& sm, RowGroup& grp, int nslots, int s0, int nl,
                                            bool wantB, bool keepP) {
    const int tid = threadIdx.x;
    slot_sums_stage1<BLK>(sm, s0, s0 + nl, wantB);
    __syncthreads();
    if (!SPLIT || grp.S == 1) {
        if (tid < nslots) {
            const double a = slot_group_sum<BLK>(sm.partA, tid);
            sm.slotA[tid] = a;
            sm.slotB[tid] = wantB ? slot_group_sum<BLK>(sm.partB, tid) : 0.0;
            if (keepP) sm.slotP[tid] = a;
        }
        __syncthreads();
        return true;
    }
    const uint32_t tag = ++grp.epoch;
    unsigned long long* xa = grp.xw + (size_t)(tag & 1u) * (2 * kMaxSlots * 2);
    unsigned long long* xb = xa + kMaxSlots * 2;
    if (tid < nl) {
        const int s = s0 + tid;
        put_tagged_d(xa + 2 * s, tag, slot_group_sum<BLK>(sm.partA, s));
        if (wantB) put_tagged_d(xb + 2 * s, tag, slot_group_sum<BLK>(sm.partB, s));
    }
    // every slot's totals, once the member that swept it has published them (the words
    // of a slot are polled together)
    int ok = 1;
    if (tid < nslots) {
        const uint64_t t0 = (uint64_t)wall_clock64();
        double a = 0.0, bv = 0.0;
        if (wantB) {
            const unsigned long long* const w[4] = {xa + 2 * tid, xa + 2 * tid + 1, xb + 2 * tid, xb + 2 * tid + 1};
            uint32_t v[4] = {0u, 0u, 0u, 0u};
            ok = get_tagged_all<4>(w, tag, v, t0, grp.wait);
            a = join_halves(v[0], v[1]);
            bv = join_halves(v[2], v[3]);
        } else {
            const unsigned long long* const w[2] = {xa + 2 * tid, xa + 2 * tid + 1};
            uint32_t v[2] = {0u, 0u};
            ok = get_tagged_all<2>(w, tag, v, t0, grp.wait);
            a = join_halves(v[0], v[1]);
        }
        sm.slotA[tid] = a;
        sm.slotB[tid] = bv;
        if (keepP) sm.slotP[tid] = a;
    }
    return __syncthreads_and(ok) != 0;
}

// Residual cache of the path schedule: two fp32 values per element of a row (the residual
// and the unnormalised draft mass), each at the element's index in a per-sequence array
// padded to a multiple of kRcPad elements (so every chunk of every layout lies inside it
// and the 16-byte accesses stay aligned).  A lane reads and writes the same VEC
// consecutive elements it takes from the logits rows.
constexpr int64_t kRcPad = 1024;

template <int VEC>
__device__ __forceinline__ void rc_load(const float* __restrict__ p, float (&v)[VEC]) {
    if constexpr (VEC % 4 == 0) {
#pragma unroll
        for (int k = 0; k < VEC / 4; ++k) {
            const float4 x = reinterpret_cast<const float4*>(p)[k];
            v[4 * k] = x.x; v[4 * k + 1] = x.y; v[4 * k + 2] = x.z; v[4 * k + 3] = x.w;
        }
    } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) v[e] = p[e];
    }
}

template <int VEC>
__device__ __forceinline__ void rc_store(float* __restrict__ p, const float (&v)[VEC]) {
    if constexpr (VEC % 4 == 0) {
#pragma unroll
        for (int k = 0; k < VEC / 4; ++k)
            reinterpret_cast<float4*>(p)[k] = make_float4(v[4 * k], v[4 * k + 1], v[4 * k + 2], v[4 * k + 3]);
    } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) p[e] = v[e];
    }
}

// One pass over the residual cache, with the slots, chunk order and wave schedule of
// wave_sweep: the residual R and the unnormalised draft mass Q of every element take the
// logits rows' place.  The sweep works in units of one load per lane and row (a chunk is
// UNR units) and keeps four unit buffers, so three units are in flight while one is
// processed; units are processed in the order they are requested.  body(r, q, i0, slot,
// u) gets R (which it may overwrite) and Q of unit u of a chunk (element e has index
// i0 + e); chunk_end(slot) runs after a chunk's last unit and flush(slot) after a slot's
// last chunk.
template <int VEC, int UNR, typename Body, typename ChunkEnd, typename Flush>
__device__ __forceinline__ void wave_sweep_rc(const float* __restrict__ rc, const float* __restrict__ qc, int G,
                                              int nslots, int sbase, bool reverse, int* counter, Body&& body,
                                              ChunkEnd&& chunk_end, Flush&& flush) {
    constexpr int CHUNK = 64 * VEC * UNR;
    const int lane = threadIdx.x & 63;
    const int wid = threadIdx.x >> 6;
    const int lane0 = lane * VEC;
    auto chunk_start = [&](int slot, int j) -> int {
        return (slot * G + (reverse ? G - 1 - j : j)) * CHUNK;
    };
    int slot = wid < nslots ? sbase + (reverse ? nslots - 1 - wid : wid) : -1;
    if (slot < 0) return;
    auto take = [&]() -> int {
        int v = 0;
        if (lane == 0) v = atomicAdd(counter, 1);
        v = __builtin_amdgcn_readfirstlane(v);
        return v < nslots ? sbase + (reverse ? nslots - 1 - v : v) : -1;
    };
    int ahead = take();
    // a unit is (slot, chunk j of the slot, load u of the chunk); slot -1: none left
    struct Unit {
        int s, j, u;
    };
    auto next = [&](Unit x) -> Unit {
        if (++x.u < UNR) return x;
        x.u = 0;
        if (++x.j < G) return x;
        x.j = 0;
        x.s = ahead;
        if (x.s >= 0) ahead = take();
        return x;
    };
    auto index = [&](const Unit& x) -> int { return chunk_start(x.s, x.j) + lane0 + x.u * 64 * VEC; };
    auto load = [&](const Unit& x, float (&r)[VEC], float (&q)[VEC]) {
        const int i0 = index(x);
        rc_load<VEC>(rc + i0, r);
        rc_load<VEC>(qc + i0, q);
    };
    auto process = [&](float (&r)[VEC], const float (&q)[VEC], const Unit& x) {
        body(r, q, index(x), x.s, x.u);
        if (x.u == UNR - 1) {
            chunk_end(x.s);
            if (x.j == G - 1) flush(x.s);
        }
    };
    float r0[VEC], r1[VEC], r2[VEC], r3[VEC];
    float q0[VEC], q1[VEC], q2[VEC], q3[VEC];
    Unit x0{slot, 0, 0};
    load(x0, r0, q0);
    Unit last = x0;
    auto refill = [&](Unit& x, float (&r)[VEC], float (&q)[VEC]) {
        if (last.s >= 0) last = next(last);
        x = last;
        if (x.s >= 0) load(x, r, q);
    };
    Unit x1, x2, x3;
    refill(x1, r1, q1);
    refill(x2, r2, q2);
    refill(x3, r3, q3);
    for (;;) {
        process(r0, q0, x0);
        refill(x0, r0, q0);
        if (x1.s < 0) break;
        process(r1, q1, x1);
        refill(x1, r1, q1);
        if (x2.s < 0) break;
        process(r2, q2, x2);
        refill(x2, r2, q2);
        if (x3.s < 0) break;
        process(r3, q3, x3);
        refill(x3, r3, q3);
        if (x0.s < 0) break;
    }
}

// How a row's draw is scheduled.  kSchedAll: every row that rejects all its candidates,
// or has none, draws at once (the all-nodes and path schedules).  kSchedDecide: a row with
// one candidate that it rejects stops after its test, keeps its pass-1 slot totals in
// P.dstate and reports RS_SEQ_DEFERRED, because the token it would draw is used only if
// a walk ends there (a row with several candidates needs its rejection passes for its
// later tests anyway, and draws at once); a leaf, whose row serves only its bonus draw,
// reports RS_SEQ_DEFERRED without reading its row.  kSchedResume: such a row is taken up
// again where its walk ends: the slot totals come from P.dstate instead of pass 1 (a leaf
// takes its pass 1 then), and every step after them is the same code on the same values,
// so the token is the one the row would have drawn at once.
constexpr int kSchedAll = 0, kSchedDecide = 1, kSchedResume = 2;
// waves whose first chunk enters the exponent reference (the waves of a 512-thread block;
// larger blocks take the same chunks, so every kernel uses the same reference)
constexpr int kRefWaves = 8;
constexpr int64_t kStateDoubles = 2 * kMaxSlots;

// A deferred row's pass-1 slot totals: the target row's, then (rows with children) the
// draft row's.
__device__ __forceinline__ void keep_slot_totals(const KParams& P, const Smem& sm, int64_t row, int nslots) {
    double* st = P.dstate + row * kStateDoubles;
    const int tid = threadIdx.x;
    if (tid < nslots) {
        st[tid] = sm.slotP[tid];
        st[kMaxSlots + tid] = sm.slotB[tid];
    }
}

// One node row's verification (the steps of Algorithm 1 at one node, or its bonus draw).
// RC: the path schedule, whose later ResiSpec rejection passes keep the row's residual
// in P.rcache when the caller's workspace holds it (see the rejection passes below).
// SCHED: how the row's draw is scheduled (above).
template <typename In, int VEC, int UNR, int MODE, int BLK, bool SPLIT, bool RC = false,
          int SCHED = kSchedAll, typename Emit>
__device__ __forceinline__ void verify_row(const KParams& P, Smem& sm, const int64_t row,
                                           const int32_t b, const int32_t n, Emit&& emit,
                                           RowGroup& grp) {
    constexpr int kBlock = BLK;
    constexpr int kWaves = BLK / 64;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int V = P.V;
    constexpr int CHUNK = 64 * VEC * UNR;
    const int G = P.G, nslots = P.nslots;
    // this workgroup's slots: all of them, or its share in a row group
    int s0 = 0, nl = nslots;
    if (SPLIT && grp.S > 1) {
        s0 = (int)((int64_t)nslots * grp.w / grp.S);
        nl = (int)((int64_t)nslots * (grp.w + 1) / grp.S) - s0;
    }

    const In* __restrict__ tg = reinterpret_cast<const In*>(P.tgt) + row * V;
    const In* __restrict__ dg = reinterpret_cast<const In*>(P.dft) + row * V;
    float* const rc = (RC && MODE == RS_MODE_RESISPEC && P.rcache) ? P.rcache + (int64_t)b * P.rc_stride : nullptr;

    using W = Vec<In, VEC>;
    if constexpr (SCHED == kSchedDecide) {
        // A leaf's row serves only its bonus draw, which is used only if a walk ends there,
        // so the row is left whole to the walk.  The tree's parent array is read first and
        // a leaf of a well-formed tree ends before any load of its row; other rows (a
        // malformed tree's included) take the description below.  Trees of up to 64 nodes
        // are read by every wave (one load a lane, no barrier), larger ones once by the
        // workgroup.  A root has a child in every well-formed tree of two or more nodes
        // (node 1's parent), so it goes straight on.
        if (!P.flat && (n > 0 || P.N == 1)) {
            const int32_t* par = P.parent + (int64_t)b * P.N;
            auto other_at = [&](int m) {   // a child of this node, or a parent entry out of place
                const int32_t pm = par[m];
                const bool bad = (m == 0) ? (pm != -1) : (pm < 0 || pm >= m);
                return bad || (m > n && pm == n);
            };
            bool leaf;
            if (P.N <= 64) {
                leaf = __ballot(lane < P.N && other_at(lane)) == 0ull;
            } else {
                int other = 0;
                for (int m = tid; m < P.N; m += kBlock) other |= other_at(m);
                leaf = !__syncthreads_or(other);
            }
            if (leaf) {
                if (tid == 0) emit(-1, -1, P.bonus ? RS_SEQ_DEFERRED : RS_SEQ_OK);
                if (!P.bonus) zero_residual_row(P, row);
                return;
            }
        }
    }
    // This wave's first target chunk is requested before the row description, so its
    // latency overlaps the description below (the first slot of wave w is slot s0 + w).
    typename W::raw pre[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) pre[u] = W::template load<kNtPass1>(tg, (s0 + wid) * G * CHUNK + lane * VEC + u * 64 * VEC, V);
    // A resumed row's stored slot totals are requested at once too (a leaf stored none;
    // its values are not used).
    double kept_a = 0.0, kept_b = 0.0;
    if constexpr (SCHED == kSchedResume) {
        if (tid < nslots) {
            const double* st = P.dstate + row * kStateDoubles;
            kept_a = st[tid];
            kept_b = st[kMaxSlots + tid];
        }
    }

    // ---- row description.  "Holder" threads own one candidate each: node, token and
    // uniform, then the two logits of its token and their unnormalised masses, all
    // written to shared memory before pass 1 starts.
    if (tid == 0) {
        sm.decision = -1;
        sm.next_slot = kWaves;
        sm.nt_hint = 0;
        sm.ur = P.flat ? P.ur_flat[row] : P.ur[row];
    }
    for (int w = tid; w < kMaxSlots / 32; w += kBlock) {
        sm.hit_slots[w] = 0u;
        sm.cand_slots[w] = 0u;
    }
    // The maximum over the first chunks of the first slots (chunk w * G for wave w < 8) fixes
    // the row's exponent reference, the same in every schedule and in every member of a
    // row group: each wave requested its chunk above, except in members whose slots start
    // later, which load those chunks' target parts here.  Elements past the row's end
    // do not count.
    auto publish_premax = [&]() {
        float mx = -FLT_MAX;
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            if (wid >= kRefWaves) break;   // the reference uses the first kRefWaves chunks
            const int idx = wid * G * CHUNK + lane * VEC + u * 64 * VEC;
            typename W::raw r = pre[u];
            if (SPLIT && s0 != 0) r = W::template load<false>(tg, idx, V);
            float v[VEC];
            W::unpack(r, v);
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                if (idx + e < V) mx = fmaxf(mx, v[e]);
        }
        mx = wave_max(mx);
        if (lane == 0) sm.wmax[0][wid] = mx;
    };
    bool holder = false;
    int32_t hx = 0, hnode = 0, hrank = 0;
    float hu = 0.0f;
    int nc = 0;
    int status = RS_SEQ_OK;
    if (P.flat) {
        holder = tid < P.k;
        if (holder) {
            hx = P.cand_ids[row * P.k + tid];
            hu = P.ua_flat[row * P.k + tid];
            hnode = tid;
            hrank = tid;
        }
        nc = P.k;
        publish_premax();
        __syncthreads();
    } else if (P.N <= kBlock) {
        const int64_t sb = (int64_t)b * P.N;
        int bad = 0;
        if (tid < P.N) {
            const int32_t pm = P.parent[sb + tid];
            hx = P.node_token[sb + tid];
            hu = P.ua[sb + tid];
            hnode = tid;
            bad = (tid == 0) ? (pm != -1) : (pm < 0 || pm >= tid);
            holder = tid > n && pm == n;
        }
        const uint64_t cm = __ballot(holder);
        const uint64_t bm = __ballot(bad);
        hrank = __popcll(cm & __lanemask_lt());
        if (lane == 0) {
            sm.wcount[wid] = __popcll(cm);
            sm.wbad[wid] = bm != 0;
        }
        publish_premax();
        __syncthreads();
        int anybad = 0;
        for (int w = 0; w < kWaves; ++w) {
            const int c = sm.wcount[w];
            nc += c;
            hrank += (w < wid) ? c : 0;
            anybad |= sm.wbad[w];
        }
        if (anybad) status = RS_SEQ_BAD_TREE;
        else if (nc > kMaxCand) status = RS_SEQ_TOO_MANY_CHILDREN;
    } else {
        // more nodes than threads: describe the row directly in shared memory
        if (tid == 0) sm.status = RS_SEQ_OK;
        publish_premax();
        const int32_t* par = P.parent + (int64_t)b * P.N;
        int bad = 0;
        for (int m = tid; m < P.N; m += kBlock) {
            const int32_t pm = par[m];
            bad |= (m == 0) ? (pm != -1) : (pm < 0 || pm >= m);
        }
        bad = __syncthreads_or(bad);
        if (wid == 0) {
            int count = 0;
            for (int base = n + 1; base < P.N; base += 64) {
                const int m = base + lane;
                const bool is_child = (m < P.N) && par[m] == n;
                const uint64_t mask = __ballot(is_child);
                if (is_child) {
                    const int idx = count + __popcll(mask & __lanemask_lt());
                    if (idx < kMaxCand) {
                        const int32_t x = P.node_token[(int64_t)b * P.N + m];
                        sm.cand_tok[idx] = x;
                        sm.cand_u[idx] = P.ua[(int64_t)b * P.N + m];
                        sm.cand_node[idx] = m;
                        const bool ok = x >= 0 && x < V;
                        sm.cand_lt[idx] = ok ? widen(tg[x]) : 0.0f;
                        sm.cand_ld[idx] = ok ? widen(dg[x]) : 0.0f;
                        if (ok && P.worep) {
                            const int cs = (x / CHUNK) / G;
                            atomicOr(&sm.cand_slots[cs >> 5], 1u << (cs & 31));
                        }
                    }
                }
                count += __popcll(mask);
            }
            if (lane == 0) {
                sm.nc = count;
                if (bad) sm.status = RS_SEQ_BAD_TREE;
                else if (count > kMaxCand) sm.status = RS_SEQ_TOO_MANY_CHILDREN;
            }
        }
        __syncthreads();
        nc = sm.nc;
        status = sm.status;
    }
    if (status != RS_SEQ_OK) {
        if (tid == 0) emit(-1, -1, status);
        zero_residual_row(P, row);
        return;
    }
    if (nc == 0 && !P.flat && !P.bonus) {
        if (tid == 0) emit(-1, -1, RS_SEQ_OK);
        zero_residual_row(P, row);
        return;
    }
    if (tid == 0) sm.status = RS_SEQ_OK;
    // candidate logits (their latency overlaps the first chunk's)
    float hlt = 0.0f, hld = 0.0f;
    if (holder && hrank < kMaxCand && hx >= 0 && hx < V) {
        hlt = widen(tg[hx]);
        hld = widen(dg[hx]);
    }

    const bool internal = nc > 0;
    if constexpr (SCHED == kSchedDecide) {
        // A row with several candidates may take many rejection passes, and the later
        // ResiSpec ones re-derive the chain of earlier steps per element (ALU-bound): such
        // rows end last.  Their waves issue ahead of the other workgroup's on the CU.
        if (nc >= 4) __builtin_amdgcn_s_setprio(3);
        else if (nc == 3) __builtin_amdgcn_s_setprio(2);
        else if (nc == 2) __builtin_amdgcn_s_setprio(1);
    }
    const float c2h = P.c2h, c2l = P.c2l;

    // ---- pass 1: softmax statistics.  Both rows are summed against one exponent
    // reference K, fixed from the maxima of the first chunks, so element values do not
    // depend on which wave read which chunk; per-lane partials of every slot go to shared
    // memory and are reduced in a fixed order.  A row whose sums overflow, or come out
    // below kLowSum, takes an exact-maximum pass and is summed again.
    float Kt, Kd;
    {
        float m0 = -FLT_MAX;
        for (int w = 0; w < kWaves; ++w) m0 = fmaxf(m0, sm.wmax[0][w]);
        Kt = Kd = kref(m0, c2h);
    }
    // The candidates' unnormalised masses need only the exponent references: holders
    // compute them (fp64) now, off the critical path after pass 1; the division by the
    // sums follows the pass.  Rows that take the exact-maximum pass recompute them.
    const double c2d = (double)c2h + (double)c2l;
    const bool holders = P.flat || P.N <= kBlock;
    bool refixed = false;
    if (holder && hrank < kMaxCand) {
        double pe = 0.0, qe = 0.0;
        if (hx >= 0 && hx < V) {
            pe = exp2((double)hlt * c2d + (double)Kt);
            qe = exp2((double)hld * c2d + (double)Kd);
            // Cache hint for pass 1 of a row with one candidate: when the candidate looks
            // accepted (its test taken with the two rows' sums assumed equal), no
            // rejection pass is expected to re-read the row, so the waves stream the rest
            // of it nontemporally.  The results do not depend on it.  When draws are
            // deferred no pass of this launch re-reads such a row, whatever its test.
            if (nc == 1 && (SCHED == kSchedDecide || (double)hu * qe < pe)) sm.nt_hint = 1;
        }
        sm.cand_tok[hrank] = hx;
        sm.cand_u[hrank] = hu;
        sm.cand_node[hrank] = hnode;
        sm.cand_lt[hrank] = hlt;
        sm.cand_ld[hrank] = hld;
        sm.cand_p[hrank] = pe;
        sm.cand_q[hrank] = qe;
        if (hx >= 0 && hx < V && P.worep) {
            const int cs = (hx / CHUNK) / G;
            atomicOr(&sm.cand_slots[cs >> 5], 1u << (cs & 31));
        }
    }
    // Without replacement pass 1 leaves the candidates out of the draft sum (their masses
    // are added in fp64 after it), so every wave needs the candidate list and its slots.
    const bool mask_cands = internal && P.worep;
    static_assert(kMaxSlots % 32 == 0 && kMaxSlots <= 128, "at most four words of candidate slots");
    constexpr int kSlotWords = kMaxSlots / 32;
    uint32_t cm0 = 0u, cm1 = 0u, cm2 = 0u, cm3 = 0u;
    if (mask_cands) {
        __syncthreads();
        cm0 = __builtin_amdgcn_readfirstlane(sm.cand_slots[0]);
        if (kSlotWords > 1) cm1 = __builtin_amdgcn_readfirstlane(sm.cand_slots[kSlotWords > 1 ? 1 : 0]);
        if (kSlotWords > 2) cm2 = __builtin_amdgcn_readfirstlane(sm.cand_slots[kSlotWords > 2 ? 2 : 0]);
        if (kSlotWords > 3) cm3 = __builtin_amdgcn_readfirstlane(sm.cand_slots[kSlotWords > 3 ? 3 : 0]);
    }
    for (int attempt = 0;; ++attempt) {
        float fa = 0.0f, fc = 0.0f;   // this slot's lane partials
        auto flush = [&](int slot) {
            sm.partA[lane][slot] = fa;
            if (internal) sm.partB[lane][slot] = fc;
            fa = fc = 0.0f;
        };
        if (SCHED == kSchedResume && internal) {
            // the slot totals pass 1 gave this row when its draw was deferred (a leaf takes
            // its pass 1 here)
            if (tid < nslots) {
                sm.slotA[tid] = kept_a;
                sm.slotP[tid] = kept_a;
                sm.slotB[tid] = kept_b;
            }
            __syncthreads();
        } else {
        if (internal) {
            wave_sweep<In, VEC, UNR, true, 1, kNtPass1>(tg, dg, V, G, nl, s0, false, pre, pre, &sm.next_slot,
                [&](const float (&t)[UNR][VEC], const float (&d)[UNR][VEC], int idx0, int slot) {
                    const int sw = slot >> 5;
                    const uint32_t cw = sw == 0 ? cm0 : (sw == 1 ? cm1 : (sw == 2 ? cm2 : cm3));
                    if ((cw >> (slot & 31)) & 1u) {
                        // a slot holding a candidate (without replacement): its draft
                        // elements are summed without the candidates.  One ballot finds
                        // the candidates inside this chunk (usually none or one).
                        const int cstart = idx0 - lane * VEC;
                        const int32_t my_cand = lane < nc ? sm.cand_tok[lane] : -1;   // lane c: candidate c
                        const uint64_t hits = __ballot(my_cand >= cstart && my_cand < cstart + CHUNK);
#pragma unroll
                        for (int u = 0; u < UNR; ++u)
#pragma unroll
                            for (int e = 0; e < VEC; ++e) {
                                fa += exp2_fast(expo(t[u][e], c2h, c2l, Kt));
                                float q = exp2_fast(expo(d[u][e], c2h, c2l, Kd));
                                const int j = idx0 + u * 64 * VEC + e;
                                for (uint64_t h = hits; h; h &= h - 1)
                                    if (j == __builtin_amdgcn_readlane(my_cand, __ffsll((long long)h) - 1)) q = 0.0f;
                                fc += q;
                            }
                        return;
                    }
#pragma unroll
                    for (int u = 0; u < UNR; ++u)
#pragma unroll
                        for (int e = 0; e < VEC; ++e) {
                            fa += exp2_fast(expo(t[u][e], c2h, c2l, Kt));
                            fc += exp2_fast(expo(d[u][e], c2h, c2l, Kd));
                        }
                },
                flush, &sm.nt_hint);
        } else if constexpr (SCHED != kSchedDecide) {   // (the decide kernel reads no leaf row)
            wave_sweep<In, VEC, UNR, false, 1, kNtLeaf, true>(tg, dg, V, G, nl, s0, false, pre, pre, &sm.next_slot,
                [&](const float (&t)[UNR][VEC], const float (&)[UNR][VEC], int, int) {
#pragma unroll
                    for (int u = 0; u < UNR; ++u)
#pragma unroll
                        for (int e = 0; e < VEC; ++e) fa += exp2_fast(expo(t[u][e], c2h, c2l, Kt));
                },
                flush);
        }
        __syncthreads();
        if (!pass_totals<BLK, SPLIT>(sm, grp, nslots, s0, nl, internal, true)) {
            if (tid == 0) emit(-1, -1, RS_SEQ_GROUP_TIMEOUT);
            zero_residual_row(P, row);
            return;
        }
        }
        if (wid == 0) {
            double a0 = 0.0, a1 = 0.0;
            for (int s2 = lane; s2 < nslots; s2 += 64) {
                a0 += sm.slotA[s2];
                a1 += sm.slotB[s2];
            }
            const double s0 = wave_sum(a0);
            const double s1 = wave_sum(a1);
            // Without replacement: the candidates' draft masses (each token once, fp64)
            // complete the draft sum, and the draft left after the first i rejections
            // weighs s1 plus the masses of the candidates from i on (a suffix sum, no
            // cancellation); its scale against the whole draft is st_ds[i].
            double wc = 0.0;
            if (mask_cands && lane < nc) {
                const int32_t x = sm.cand_tok[lane];
                bool first = x >= 0 && x < V;
                for (int c = 0; c < lane; ++c) first = first && sm.cand_tok[c] != x;
                if (first) wc = exp2((double)sm.cand_ld[lane] * c2d + (double)Kd);
            }
            const double sd = mask_cands ? s1 + wave_sum(wc) : s1;
            const bool ok = s0 >= kLowSum && s0 < INFINITY && (!internal || (sd >= kLowSum && sd < INFINITY));
            if (mask_cands) {
                double suf = 0.0;
                for (int c = nc - 1; c >= 0; --c) {
                    suf += readlane_d(wc, c);
                    const double rem = s1 + suf;
                    if (lane == 0) sm.st_ds[c] = c == 0 ? 1.0 : (rem > 0.0 ? sd / rem : 0.0);
                }
                if (lane == 0) sm.st_ds[nc] = s1 > 0.0 ? sd / s1 : 0.0;
            } else if (lane == 0) {
                for (int c = 0; c <= nc; ++c) sm.st_ds[c] = 1.0;
            }
            if (lane == 0) {
                sm.St = s0;
                sm.Sd = sd;
                sm.Sd_nc = s1;
                sm.decision = ok ? -1 : -3;   // -3: sum again with exact maxima
                sm.next_slot = kWaves;
            }
        }
        __syncthreads();
        if (sm.decision != -3) break;
        if (attempt == 1) {
            if (tid == 0) emit(-1, -1, RS_SEQ_UNDERFLOW);
            zero_residual_row(P, row);
            return;
        }
        // exact maxima of both rows, then the references are taken from them
        {
            float mx = -FLT_MAX, my = -FLT_MAX;
            wave_sweep<In, VEC, UNR, true, 0, kNtPass1>(tg, dg, V, G, nl, s0, false, pre, pre, &sm.next_slot,
                [&](const float (&t)[UNR][VEC], const float (&d)[UNR][VEC], int, int) {
#pragma unroll
                    for (int u = 0; u < UNR; ++u)
#pragma unroll
                        for (int e = 0; e < VEC; ++e) {
                            mx = fmaxf(mx, t[u][e]);
                            my = internal ? fmaxf(my, d[u][e]) : my;
                        }
                },
                [](int) {});
            mx = wave_max(mx);
            my = wave_max(my);
            if (lane == 0) {
                sm.wmax[0][wid] = mx;
                sm.wmax[1][wid] = my;
            }
            __syncthreads();
            float m0 = -FLT_MAX, m1 = -FLT_MAX;
            for (int w = 0; w < kWaves; ++w) {
                m0 = fmaxf(m0, sm.wmax[0][w]);
                m1 = fmaxf(m1, sm.wmax[1][w]);
            }
            if (SPLIT && grp.S > 1) {   // the maxima of the whole row, from every member
                const uint32_t tag = ++grp.epoch;
                unsigned long long* xm = grp.xm + (size_t)(tag & 1u) * (kMaxGroup * 2);
                if (tid == 0) {
                    put_tagged(xm + 2 * grp.w, tag, __float_as_uint(m0));
                    put_tagged(xm + 2 * grp.w + 1, tag, __float_as_uint(m1));
                }
                __syncthreads();   // every thread has read the waves' maxima
                int ok = 1;
                if (tid < grp.S) {
                    const uint64_t t0 = (uint64_t)wall_clock64();
                    uint32_t v0 = 0, v1 = 0;
                    const unsigned long long* const wm[2] = {xm + 2 * tid, xm + 2 * tid + 1};
                    uint32_t vm[2] = {0u, 0u};
                    ok = get_tagged_all<2>(wm, tag, vm, t0, grp.wait);
                    v0 = vm[0];
                    v1 = vm[1];
                    sm.wmax[0][tid] = __uint_as_float(v0);
                    sm.wmax[1][tid] = __uint_as_float(v1);
                }
                if (!__syncthreads_and(ok)) {
                    if (tid == 0) emit(-1, -1, RS_SEQ_GROUP_TIMEOUT);
                    zero_residual_row(P, row);
                    return;
                }
                m0 = m1 = -FLT_MAX;
                for (int q = 0; q < grp.S; ++q) {
                    m0 = fmaxf(m0, sm.wmax[0][q]);
                    m1 = fmaxf(m1, sm.wmax[1][q]);
                }
            }
            Kt = kref(m0, c2h);
            Kd = kref(m1, c2h);
            refixed = true;
            if (tid == 0) {
                sm.decision = -1;
                sm.next_slot = kWaves;
            }
            __syncthreads();
        }
    }

    // Deferred draws: a row with one candidate that it rejects keeps its pass-1 slot totals
    // and reports RS_SEQ_DEFERRED.  Rows that took the exact-maximum pass draw at once
    // (their exponent references are not the ones a resumed row derives).
    const bool deferrable = SCHED == kSchedDecide && !P.flat && !refixed;

    const double St = sm.St, Sd = sm.Sd;
    // draft mass in target units: q St / Sd, folded into the step constants
    const double q2t = internal ? St / Sd : 0.0;

    // ---- candidate probabilities in fp64, with the same exponent constants
    if (tid < nc) {
        const int32_t x = sm.cand_tok[tid];
        double pc = 0.0, qc = 0.0;
        if (x >= 0 && x < V) {
            const bool early = holders && !refixed;
            const double pe = early ? sm.cand_p[tid] : exp2((double)sm.cand_lt[tid] * c2d + (double)Kt);
            const double qe = early ? sm.cand_q[tid] : exp2((double)sm.cand_ld[tid] * c2d + (double)Kd);
            pc = pe / St;
            qc = qe / Sd;
        }
        sm.cand_p[tid] = pc;
        sm.cand_q[tid] = qc;
    }
    __syncthreads();

    const bool worep = P.worep != 0;

    // ---- sequential accept / reject
    int i = 0;
    for (; i < nc; ++i) {
        if (tid == 0) {
            const int32_t x = sm.cand_tok[i];
            const float u = sm.cand_u[i];
            int dec = -1;
            if (x < 0 || x >= V) {
                sm.status = RS_SEQ_BAD_TOKEN;
                dec = -2;
            } else if (!(u >= 0.0f && u < 1.0f)) {
                sm.status = RS_SEQ_BAD_UNIFORM;
                dec = -2;
            } else {
                const ResDraft rd = scalar_residual<MODE>(sm, i, sm.cand_p[i], sm.cand_q[i], x, worep);
                const double Rx = rd.R, Dx = rd.D;
                if (!(Dx > 0.0)) {
                    sm.status = RS_SEQ_ZERO_DRAFT;
                    dec = -2;
                } else if ((double)u < Rx / Dx) {
                    dec = i;
                } else {
                    const double z = Dx - Rx;   // ResiSpec budget
                    sm.st_x[i] = x;
                    sm.st_rx[i] = Rx;
                    const int hs = (x / CHUNK) / G;
                    sm.hit_slots[hs >> 5] |= 1u << (hs & 31);
                    sm.st_zd[i] = z;
                    if (MODE == RS_MODE_SPECINFER) {
                        const double C = (i == 0) ? sm.st_ds[0]
                                                  : sm.st_C[i - 1] + sm.st_tot[i - 1] * sm.st_ds[i];
                        sm.st_C[i] = C;
                        sm.st_c[i] = (float)(C * q2t);
                    } else {
                        const double c = z * sm.st_ds[i] * q2t;
                        sm.st_c[i] = (float)c;
                        if (i == 0) {
                            // c = m 2^e exactly, m in [0.5, 1); log2 m in fp32.  The split
                            // only has to reproduce c to fp32 accuracy, like st_c itself.
                            int e;
                            const double m = frexp(c, &e);
                            const float f0 = __builtin_amdgcn_logf((float)m);
                            sm.st_f0 = f0;
                            sm.st_kq0 = Kd + (float)e;
                            sm.st_2f0 = (double)exp2_fast(f0);
                            sm.rx0e = (double)exp2_fast(expo(sm.cand_lt[0], c2h, c2l, Kt));
                            sm.sx0 = hs;
                        }
                    }
                    sm.next_slot = kWaves;
                }
            }
            sm.decision = dec;
        }
        __syncthreads();
        if (sm.decision != -1) break;
        // one candidate, rejected: the draw from the residual is used only if a walk ends here
        if constexpr (SCHED == kSchedDecide) {
            if (deferrable && nc == 1) {
                keep_slot_totals(P, sm, row, nslots);
                if (tid == 0) emit(-1, -1, RS_SEQ_DEFERRED);
                return;
            }
        }

        // rejection pass: sums of step i with per-slot partials
        {
            float accA = 0.0f, accB = 0.0f;   // this slot's lane partials
            const bool reverse = (i & 1) == 0;   // re-read the most recently fetched end first
            const int ii = i;
            const float ci = sm.st_c[i];
            const int xi = sm.st_x[i];
            // ResiSpec needs the per-slot sums of R only after the first rejection
            const bool wantB = MODE == RS_MODE_RESISPEC && ii > 0;
            auto flush = [&](int slot) {
                sm.partA[lane][slot] = accA;
                if (wantB) sm.partB[lane][slot] = accB;
                accA = accB = 0.0f;
            };
            // Load policy.  In the decide kernel only rows with several candidates take
            // rejection passes, and while a candidate is left the row is read again: the
            // passes keep it in the caches, as do the path schedule's with its residual
            // cache (its second pass reads the logits again).  Elsewhere a rejection pass is
            // mostly the row's last use and streams nontemporally.
            constexpr bool kNtRejPass = (SCHED == kSchedDecide || RC) ? false : kNtRej;
            // does this slot hold a rejected token? (wave-uniform)
            auto slot_hit = [&](int slot) -> bool {
                const uint32_t w = __builtin_amdgcn_readfirstlane(sm.hit_slots[slot >> 5]);
                return (w >> (slot & 31)) & 1u;
            };
            if (MODE == RS_MODE_SPECINFER) {
                // A = max(R - C_i Q, 0)
                wave_sweep<In, VEC, UNR, true, 0, kNtRejPass>(tg, dg, V, G, nl, s0, reverse, pre, pre, &sm.next_slot,
                    [&](const float (&t)[UNR][VEC], const float (&d)[UNR][VEC], int, int) {
                        float fa = 0.0f;
#pragma unroll
                        for (int u = 0; u < UNR; ++u)
#pragma unroll
                            for (int e = 0; e < VEC; ++e) {
                                const float R = exp2_fast(expo(t[u][e], c2h, c2l, Kt));
                                const float Q = exp2_fast(expo(d[u][e], c2h, c2l, Kd));
                                fa += fmaxf(fmaf(-ci, Q, R), 0.0f);
                            }
                        accA += fa;
                    },
                    flush);
            } else if (ii == 0) {
                // first rejection: A = min(c Q, R) / 2^f0 = exp2(min(aR - f0, aQ + e)), one
                // exponential per element; the sum of R over j != x_0 is 1 - R(x_0)
                const float f0 = sm.st_f0, kq0 = sm.st_kq0;
                wave_sweep<In, VEC, UNR, true, 0, kNtRejPass>(tg, dg, V, G, nl, s0, reverse, pre, pre, &sm.next_slot,
                    [&](const float (&t)[UNR][VEC], const float (&d)[UNR][VEC], int idx0, int slot) {
                        float v[UNR][VEC];
#pragma unroll
                        for (int u = 0; u < UNR; ++u)
#pragma unroll
                            for (int e = 0; e < VEC; ++e)
                                v[u][e] = exp2_fast(fminf(expo(t[u][e], c2h, c2l, Kt) - f0,
                                                          expo(d[u][e], c2h, c2l, kq0)));
                        if (slot_hit(slot)) {
#pragma unroll
                            for (int u = 0; u < UNR; ++u)
#pragma unroll
                                for (int e = 0; e < VEC; ++e)
                                    if (idx0 + u * 64 * VEC + e == xi) v[u][e] = 0.0f;
                        }
                        float fa = 0.0f;
#pragma unroll
                        for (int u = 0; u < UNR; ++u)
#pragma unroll
                            for (int e = 0; e < VEC; ++e) fa += v[u][e];
                        accA += fa;
                    },
                    flush);
            } else if (RC && rc) {
                // Later rejections with the residual cache.  Pass i applies step i - 1 of
                // the chain to the residual the previous pass left in the cache (pass 1
                // starts from the target row), stores the result for the next pass when
                // a candidate is left, and sums as below: one step per element instead of
                // i, with the same fp32 operations in the same order as the chain, so the
                // values are bit for bit those of the other schedules.  Pass 1 also
                // stores the draft masses Q, so the later passes read no logits and take
                // no exponentials.
                const float kc = sm.st_kc[ii - 1], k1 = sm.st_k1[ii - 1], inv = sm.st_i[ii - 1];
                const int xp = sm.st_x[ii - 1];
                const bool keep = ii + 1 < nc;
                const int64_t rcq = P.rc_stride / 2;   // Q's half of the sequence's cache
                // one load's elements (u) at a time; the sums add them in the chain's order
                auto step = [&](float (&R)[VEC], const float (&Q)[VEC], int i0, bool hit, float& fa, float& fb) {
#pragma unroll
                    for (int e = 0; e < VEC; ++e) R[e] = fminf(fmaf(kc, Q[e], k1 * R[e]), inv * R[e]);
                    if (hit) {
#pragma unroll
                        for (int e = 0; e < VEC; ++e)
                            if (i0 + e == xp) R[e] = 0.0f;
                    }
                    if (keep) rc_store<VEC>(rc + i0, R);
                    if (keep && ii == 1) rc_store<VEC>(rc + rcq + i0, Q);
                    if (hit) {
#pragma unroll
                        for (int e = 0; e < VEC; ++e)
                            if (i0 + e == xi) R[e] = 0.0f;
                    }
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        fa += fminf(ci * Q[e], R[e]);
                        fb += R[e];
                    }
                };
                if (ii == 1) {
                    wave_sweep<In, VEC, UNR, true, 0, kNtRejPass>(tg, dg, V, G, nl, s0, reverse, pre, pre, &sm.next_slot,
                        [&](const float (&t)[UNR][VEC], const float (&d)[UNR][VEC], int idx0, int slot) {
                            const bool hit = slot_hit(slot);
                            float fa = 0.0f, fb = 0.0f;
#pragma unroll
                            for (int u = 0; u < UNR; ++u) {
                                float R[VEC], Q[VEC];
#pragma unroll
                                for (int e = 0; e < VEC; ++e) {
                                    R[e] = exp2_fast(expo(t[u][e], c2h, c2l, Kt));
                                    Q[e] = exp2_fast(expo(d[u][e], c2h, c2l, Kd));
                                }
                                step(R, Q, idx0 + u * 64 * VEC, hit, fa, fb);
                            }
                            accA += fa;
                            accB += fb;
                        },
                        flush);
                } else {
                    // the chunk's sums run across its units in the order above
                    float fa = 0.0f, fb = 0.0f;
                    bool hit = false;   // the chunk's slot holds a rejected token (read at its first unit)
                    wave_sweep_rc<VEC, UNR>(rc, rc + rcq, G, nl, s0, reverse, &sm.next_slot,
                        [&](float (&r)[VEC], const float (&q)[VEC], int i0, int slot, int u) {
                            if (u == 0) hit = slot_hit(slot);
                            step(r, q, i0, hit, fa, fb);
                        },
                        [&](int) {
                            accA += fa;
                            accB += fb;
                            fa = fb = 0.0f;
                        },
                        flush);
                }
            } else {
                wave_sweep<In, VEC, UNR, true, 0, kNtRejPass>(tg, dg, V, G, nl, s0, reverse, pre, pre, &sm.next_slot,
                    [&](const float (&t)[UNR][VEC], const float (&d)[UNR][VEC], int idx0, int slot) {
                        const bool hit = slot_hit(slot);
                        float R[UNR][VEC], Q[UNR][VEC];
#pragma unroll
                        for (int u = 0; u < UNR; ++u)
#pragma unroll
                            for (int e = 0; e < VEC; ++e) {
                                R[u][e] = exp2_fast(expo(t[u][e], c2h, c2l, Kt));
                                Q[u][e] = exp2_fast(expo(d[u][e], c2h, c2l, Kd));
                            }
                        for (int s2 = 0; s2 < ii; ++s2) {
                            const float kc = sm.st_kc[s2], k1 = sm.st_k1[s2], inv = sm.st_i[s2];
#pragma unroll
                            for (int u = 0; u < UNR; ++u)
#pragma unroll
                                for (int e = 0; e < VEC; ++e)
                                    R[u][e] = fminf(fmaf(kc, Q[u][e], k1 * R[u][e]), inv * R[u][e]);
                            if (hit) {
                                const int x = sm.st_x[s2];
#pragma unroll
                                for (int u = 0; u < UNR; ++u)
#pragma unroll
                                    for (int e = 0; e < VEC; ++e)
                                        if (idx0 + u * 64 * VEC + e == x) R[u][e] = 0.0f;
                            }
                        }
                        if (hit) {
#pragma unroll
                            for (int u = 0; u < UNR; ++u)
#pragma unroll
                                for (int e = 0; e < VEC; ++e)
                                    if (idx0 + u * 64 * VEC + e == xi) R[u][e] = 0.0f;
                        }
                        float fa = 0.0f, fb = 0.0f;
#pragma unroll
                        for (int u = 0; u < UNR; ++u)
#pragma unroll
                            for (int e = 0; e < VEC; ++e) {
                                fa += fminf(ci * Q[u][e], R[u][e]);
                                fb += R[u][e];
                            }
                        accA += fa;
                        accB += fb;
                    },
                    flush);
            }
        }
        __syncthreads();
        if (!pass_totals<BLK, SPLIT>(sm, grp, nslots, s0, nl, MODE == RS_MODE_RESISPEC && i > 0, false)) {
            if (tid == 0) emit(-1, -1, RS_SEQ_GROUP_TIMEOUT);
            zero_residual_row(P, row);
            return;
        }
        if (wid == 0) {
            // per-lane sums over slots lane, lane+64, ... in a fixed order
            double A = 0.0, Bv = 0.0;
            for (int s2 = lane; s2 < nslots; s2 += 64) {
                A += sm.slotA[s2];
                Bv += sm.slotB[s2];
            }
            const double z = sm.st_zd[i];
            if (MODE == RS_MODE_SPECINFER) {
                const double tot = wave_sum(A) / St;   // normalised units
                if (lane == 0) {
                    if (!(tot > 0.0)) {
                        sm.status = RS_SEQ_UNDERFLOW;
                        sm.decision = -2;
                    }
                    sm.st_tot[i] = tot;
                }
                for (int s2 = lane; s2 < nslots; s2 += 64) sm.slotT[s2] = sm.slotA[s2];
            } else {
                // GetProxy: M = sum min(Z D, R), SR = sum R (both over j != x_i),
                // a = (Z - M) / (SR - M)
                const double scale = (i == 0) ? sm.st_2f0 : 1.0;
                const double M = wave_sum(A) * scale / St;
                const double SR = (i == 0) ? 1.0 - sm.st_rx[0] : wave_sum(Bv) / St;
                const double C = SR - M;                 // remaining capacity, x0 excluded
                const double a = (C > 0.0) ? (z - M) / C : 0.0;
                // slot totals of the unnormalised next residual (linear in the partials);
                // after the first rejection the slot sums of R are the pass-1 totals
                // without x_0
                for (int s2 = lane; s2 < nslots; s2 += 64) {
                    double Bs = sm.slotB[s2];
                    if (i == 0) {
                        Bs = sm.slotP[s2] - (s2 == sm.sx0 ? sm.rx0e : 0.0);
                        Bs = Bs > 0.0 ? Bs : 0.0;
                    }
                    sm.slotT[s2] = (1.0 - a) * sm.slotA[s2] * scale + a * Bs;
                }
                if (lane == 0) {
                    sm.st_ad[i] = a;
                    sm.st_a[i] = (float)a;
                    sm.st_i[i] = (float)(1.0 / z);
                    sm.st_k1[i] = (float)(a / z);
                    sm.st_kc[i] = (float)((1.0 - a) * sm.st_ds[i] * q2t);   // (1 - a) c / Z
                }
            }
        }
        __syncthreads();
        if (sm.decision == -2) break;
    }

    if (sm.decision == -2) {
        if (tid == 0) emit(-1, -1, sm.status);
        zero_residual_row(P, row);
        return;
    }
    if (sm.decision >= 0) {
        if (tid == 0) {
            const int d = sm.decision;
            emit(sm.cand_node[d], sm.cand_tok[d], RS_SEQ_OK);
        }
        zero_residual_row(P, row);
        return;
    }

    // ---- every candidate rejected, or no candidates: inverse-CDF draw (wave 0)
    const float u = sm.ur;
    if (!(u >= 0.0f && u < 1.0f)) {
        if (tid == 0) emit(-1, -1, RS_SEQ_BAD_UNIFORM);
        zero_residual_row(P, row);
        return;
    }
    const int last = nc - 1;   // index of the last rejection step (internal rows)
    const float a_last = (internal && MODE == RS_MODE_RESISPEC) ? sm.st_a[last] : 0.0f;
    const bool first_only = internal && MODE == RS_MODE_RESISPEC && last == 0;
    const float f0 = first_only ? sm.st_f0 : 0.0f, kq0 = first_only ? sm.st_kq0 : 0.0f;
    const float s2f0 = first_only ? (float)sm.st_2f0 : 0.0f;
    const int32_t x0 = first_only ? sm.st_x[0] : -1;
    // element values of the final distribution (unnormalised, target units), computed
    // as in the pass that produced the slot totals
    auto final_value = [&](float lt, float ld, int j) -> float {
        const float R = exp2_fast(expo(lt, c2h, c2l, Kt));
        if (!internal) return R;
        if (first_only) {
            if (j == x0) return 0.0f;
            const float A = s2f0 * exp2_fast(fminf(expo(lt, c2h, c2l, Kt) - f0, expo(ld, c2h, c2l, kq0)));
            return fmaf(a_last, R - A, A);
        }
        const float Q = exp2_fast(expo(ld, c2h, c2l, Kd));
        float A, Bv;
        chain_terms<MODE>(R, Q, j, sm, last, A, Bv);
        if (MODE == RS_MODE_SPECINFER) return A;
        return fmaf(a_last, Bv - A, A);
    };
    // The same values for VEC consecutive elements from j0: the chain's per-step constants
    // are read once per step for all of them (each element takes the operations of
    // final_value, in the same order).
    auto final_values = [&](const float (&lt)[VEC], const float (&ld)[VEC], int j0, float (&out)[VEC]) {
        if (!internal || first_only) {
#pragma unroll
            for (int e = 0; e < VEC; ++e) out[e] = final_value(lt[e], ld[e], j0 + e);
            return;
        }
        float R[VEC], Q[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            R[e] = exp2_fast(expo(lt[e], c2h, c2l, Kt));
            Q[e] = exp2_fast(expo(ld[e], c2h, c2l, Kd));
        }
        if (MODE == RS_MODE_SPECINFER) {
            const float ci = sm.st_c[last];
#pragma unroll
            for (int e = 0; e < VEC; ++e) out[e] = fmaxf(fmaf(-ci, Q[e], R[e]), 0.0f);
            return;
        }
        for (int t = 0; t < last; ++t) {
            const float kc = sm.st_kc[t], k1 = sm.st_k1[t], inv = sm.st_i[t];
            const int32_t xt = sm.st_x[t];
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                R[e] = fminf(fmaf(kc, Q[e], k1 * R[e]), inv * R[e]);
                if (j0 + e == xt) R[e] = 0.0f;
            }
        }
        const float ci = sm.st_c[last];
        const int32_t xl = sm.st_x[last];
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            const bool at = j0 + e == xl;
            const float A = at ? 0.0f : fminf(ci * Q[e], R[e]);
            const float Bv = at ? 0.0f : R[e];
            out[e] = fmaf(a_last, Bv - A, A);
        }
    };
    if (wid == 0) {
        // slot totals in vocabulary order; lane l holds slots 4l .. 4l+3
        double Ts[4];
        double own = 0.0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int s2 = 4 * lane + q;
            double T = 0.0;
            if (s2 < nslots) T = internal ? sm.slotT[s2] : sm.slotA[s2];
            Ts[q] = T;
            own += T;
        }
        const double incl = wave_incl_scan(own, lane);
        const double total = readlane_d(incl, 63);
        const double thr = (double)u * total;
        const double excl = incl - own;
        uint64_t hit = __ballot(own > 0.0 && incl > thr);
        int L = hit ? (__ffsll((unsigned long long)hit) - 1) : -1;
        if (L < 0) {   // rounding guard: last lane with mass
            const uint64_t pos = __ballot(own > 0.0);
            L = pos ? 63 - __clzll((long long)pos) : 0;
        }
        int ks = -1;
        double base = 0.0;
        if (lane == L) {
            double c = excl;
            int lastpos = -1;
            double lastbase = 0.0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                if (Ts[q] > 0.0) {
                    if (ks < 0 && c + Ts[q] > thr) {
                        ks = 4 * lane + q;
                        base = c;
                    }
                    lastpos = 4 * lane + q;
                    lastbase = c;
                }
                c += Ts[q];
            }
            if (ks < 0) {
                ks = lastpos;
                base = lastbase;
            }
        }
        ks = __builtin_amdgcn_readlane(ks, L);
        base = readlane_d(base, L);
        if (ks < 0) {   // no mass anywhere (degenerate): no draw
            if (lane == 0) {
                sm.token = -1;
                sm.total = total;
                sm.status = RS_SEQ_UNDERFLOW;
            }
        } else {
        // the slot's elements: lane l takes a contiguous run of R = G * VEC * UNR
        const int R = G * VEC * UNR;
        const int t0 = ks * G * CHUNK + lane * R;
        double own2 = 0.0;
        // The run's values are staged in the lane's row of the pass partials (idle during
        // the draw) when the run fits there; one chunk's loads stay in flight ahead of the
        // arithmetic.  A rolled loop keeps the kernel's code small: fully unrolled, the
        // value code of every element made the kernel larger than the instruction cache.
        const bool staged = R <= kMaxSlots;
        {
            float tv[VEC], dv[VEC];
            load_vec<In, VEC>(tg, t0, V, tv);
            if (internal) load_vec<In, VEC>(dg, t0, V, dv);
#pragma unroll 1
            for (int c = 0; c < R; c += VEC) {
                float tn[VEC], dn[VEC];
                const bool more = c + VEC < R;
                if (more) {
                    load_vec<In, VEC>(tg, t0 + c + VEC, V, tn);
                    if (internal) load_vec<In, VEC>(dg, t0 + c + VEC, V, dn);
                }
                float vals[VEC];
                if (!internal) {
#pragma unroll
                    for (int e = 0; e < VEC; ++e) dv[e] = 0.0f;
                }
                final_values(tv, dv, t0 + c, vals);
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    const int j = t0 + c + e;
                    const float v = j < V ? vals[e] : 0.0f;
                    if (staged) sm.partA[lane][c + e] = v;
                    own2 += (double)v;
                }
                if (more) {
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        tv[e] = tn[e];
                        if (internal) dv[e] = dn[e];
                    }
                }
            }
        }
        const double incl2 = wave_incl_scan(own2, lane);
        const double excl2 = incl2 - own2;
        const uint64_t hit2 = __ballot(own2 > 0.0 && base + incl2 > thr);
        int L2 = hit2 ? (__ffsll((unsigned long long)hit2) - 1) : -1;
        const bool fallback = L2 < 0;
        if (fallback) {   // rounding guard: last lane of the slot with mass
            const uint64_t pos = __ballot(own2 > 0.0);
            L2 = pos ? 63 - __clzll((long long)pos) : -1;
        }
        if (lane == L2) {
            double acc = base + excl2;
            int tok = -1, lastpos = -1;
            if (staged) {
#pragma unroll 1
                for (int c = 0; c < R && tok < 0; ++c) {
                    const int j = t0 + c;
                    if (j >= V) break;
                    const float v = sm.partA[lane][c];
                    if (v > 0.0f) lastpos = j;
                    acc += (double)v;
                    if (!fallback && v > 0.0f && acc > thr) tok = j;
                }
            } else {
                for (int c = 0; c < R && tok < 0; c += VEC) {
                    float tv[VEC], dv[VEC];
                    load_vec<In, VEC>(tg, t0 + c, V, tv);
                    if (internal) load_vec<In, VEC>(dg, t0 + c, V, dv);
                    for (int e = 0; e < VEC; ++e) {
                        const int j = t0 + c + e;
                        if (j >= V) break;
                        const float v = final_value(tv[e], internal ? dv[e] : 0.0f, j);
                        if (v > 0.0f) lastpos = j;
                        acc += (double)v;
                        if (!fallback && v > 0.0f && acc > thr) {
                            tok = j;
                            break;
                        }
                    }
                }
            }
            if (tok < 0) tok = lastpos;
            sm.token = tok;
        }
        if (lane == 0) {
            if (L2 < 0) sm.token = -1;
            sm.total = total;
            if (!(total > 0.0)) sm.status = RS_SEQ_UNDERFLOW;
        }
        }
    }
    __syncthreads();
    const int32_t tok = sm.token;
    if (tid == 0) {
        if (sm.status != RS_SEQ_OK) emit(-1, -1, sm.status);
        else if (tok < 0) emit(-1, -1, RS_SEQ_UNDERFLOW);
        else emit(-1, tok, RS_SEQ_OK);
    }

    // debug: the normalised distribution of the draw
    if (P.residual_out) {
        float* out = P.residual_out + row * V;
        const double inv_total = 1.0 / sm.total;
        for (int j = tid; j < V; j += kBlock) {
            const float lt = widen(tg[j]);
            const float ld = internal ? widen(dg[j]) : 0.0f;
            out[j] = (float)((double)final_value(lt, ld, j) * inv_total);
        }
    }
}


// One workgroup per node row; the grid is node-major: the roots of all sequences first,
// then node 1, ... (nodes with children, whose rows take rejection passes, come early
// in a topological numbering, so the grid ends on short rows; an order that mixes
// sequences' rows runs 1.5x longer on a 128-tree batch because late roots form a tail).
template <typename In, int VEC, int UNR, int MODE>
__global__ void __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) rs_row_kernel(const KParams P) {
    __shared__ Smem sm;
    int64_t row;
    int32_t b, n;
    if (P.flat) {
        row = blockIdx.x;
        b = (int32_t)row;
        n = 0;
    } else {
        const int32_t g = blockIdx.x;
        n = g / P.B;
        b = g - n * P.B;
        row = (int64_t)b * P.N + n;
    }
    RowGroup solo{1, 0, nullptr, nullptr, 0u, kGroupWaitTicks};
    verify_row<In, VEC, UNR, MODE, kBlock, false>(P, sm, row, b, n, [&](int32_t child, int32_t tok, int32_t st) {
        write_outcome(P, row, child, tok, st);
    }, solo);
}

// Row groups: S members per sequence (path schedule) or per row (all-nodes schedule),
// the workspace that holds each group's state (kGroupStride bytes per group), and the
// time limits; group_of below says which workgroup is which member.  S = 1 needs no
// workspace.
struct GroupArgs {
    int32_t S;
    char* ws;
    uint64_t wait;       // exchange time limit (ticks)
    uint64_t form_wait;  // formation time limit (ticks)
    int32_t groups;      // groups with work (sequences or rows)
    int32_t xcd;         // 1: the XCD layout below
};

// Which group and member a workgroup is.  The dispatcher deals the workgroups of a launch
// round-robin over the 8 XCDs (workgroup i runs on XCD i % 8), and each XCD has its own
// L2.  In the XCD layout the S members of group g all run on XCD g % 8, so the traffic
// of their exchanges stays within one L2: workgroup i = 8 k + x is member
// k % S of group x + 8 (k / S).  The grid then holds a multiple of 8 groups, and the
// workgroups of groups past the last return at once.  Without it, workgroup i is member
// i % S of group i / S.  Returns false for a padding workgroup.
__device__ __forceinline__ bool group_of(const GroupArgs& ga, int32_t& g, int32_t& w) {
    const uint32_t i = blockIdx.x, S = (uint32_t)ga.S;
    if (ga.xcd) {
        const uint32_t k = i >> 3;
        g = (int32_t)((i & 7u) + 8u * (k / S));
        w = (int32_t)(k % S);
    } else {
        g = (int32_t)(i / S);
        w = (int32_t)(i % S);
    }
    return g < ga.groups;
}

// Path-only schedule: a sequence's workgroup (or row group) walks its own tree from the
// root and verifies only the nodes it reaches (each node's outcome depends on that
// node's rows and uniforms alone, so the result equals the all-nodes schedule followed
// by the walk, bit for bit: rows are cut into the same chunks and slots, and summed in
// the same order).  Member 0 of a group (or the member that claimed the sequence)
// writes the outputs.  The walk keeps its state
// live across every row, so these workgroups take up to 256 registers per lane (two
// waves per SIMD, one workgroup per CU) and nothing is spilled.
constexpr int kPathBlock = 512;
constexpr int kPathAutoSlots = 4;   // automatic path row groups: at least this many slots a member

template <typename In, int VEC, int UNR, int MODE>
__global__ void __launch_bounds__(kPathBlock) __attribute__((amdgpu_waves_per_eu(2)))
rs_path_kernel(const KParams P, int32_t max_depth, int32_t* __restrict__ out_tokens,
               int32_t* __restrict__ out_len, int32_t* __restrict__ out_status, const GroupArgs ga) {
    constexpr int kBlock = kPathBlock;
    __shared__ Smem sm;
    const int tid = threadIdx.x;
    const int32_t S = ga.S;
    int32_t b, member;
    if (!group_of(ga, b, member)) return;
    RowGroup grp{S, member, nullptr, nullptr, 0u, ga.wait};
    bool lead = member == 0;
    if (S > 1) {
        char* base = ga.ws + (int64_t)b * kGroupStride;
        grp.xw = reinterpret_cast<unsigned long long*>(base + kGroupXw);
        grp.xm = reinterpret_cast<unsigned long long*>(base + kGroupXm);
        const int form = form_group(sm, grp, base, ga.form_wait);
        if (form == 0) return;   // another member does this sequence's walk alone
        if (form == 2) {         // this member does it alone: every slot, no exchanges
            grp.S = 1;
            grp.w = 0;
            lead = true;
        }
    }
    const int32_t N = P.N;
    const int64_t W = (int64_t)max_depth + 1;
    int32_t* out = out_tokens + (int64_t)b * W;
    if (lead)
        for (int64_t i = tid; i < W; i += kBlock) out[i] = -1;
    int32_t n = 0, len = 0, status = RS_SEQ_OK;
    for (int32_t steps = 0; steps <= N; ++steps) {
        verify_row<In, VEC, UNR, MODE, kBlock, true, true>(P, sm, (int64_t)b * N + n, b, n,
                                                     [&](int32_t child, int32_t tok, int32_t st) {
            sm.res_child = child;
            sm.res_tok = tok;
            sm.res_status = st;
        }, grp);
        __syncthreads();
        const int32_t st = __builtin_amdgcn_readfirstlane(sm.res_status);
        const int32_t c = __builtin_amdgcn_readfirstlane(sm.res_child);
        const int32_t t = __builtin_amdgcn_readfirstlane(sm.res_tok);
        __syncthreads();   // the next row rewrites the shared state
        if (st != RS_SEQ_OK) {
            status = st;
            break;
        }
        if (c >= 0) {
            if (c <= n || c >= N) {
                status = RS_SEQ_BAD_TREE;
                break;
            }
            if (len >= max_depth) {
                status = RS_SEQ_DEPTH_EXCEEDED;
                break;
            }
            if (lead && tid == 0) out[len] = P.node_token[(int64_t)b * N + c];
            ++len;
            n = c;
            continue;
        }
        if (t >= 0 && lead && tid == 0) out[len] = t;
        break;
    }
    if (status != RS_SEQ_OK) {
        __syncthreads();
        if (lead)
            for (int64_t i = tid; i < W; i += kBlock) out[i] = -1;
        len = -1;
    }
    if (lead && tid == 0) {
        out_len[b] = len;
        if (out_status) out_status[b] = status;
    }
}

// A row group's formation counters and exchange words start at zero in every launch (one
// group state of kGroupStride bytes per sequence or per row; a block of 256 threads per
// group).
constexpr int kResetBlock = 256;
__global__ void __launch_bounds__(kResetBlock) rs_group_reset(char* __restrict__ ws, int32_t count) {
    const int64_t g = blockIdx.x;
    if (g >= count) return;
    char* base = ws + g * kGroupStride;
    if (threadIdx.x == 0) {
        *reinterpret_cast<uint32_t*>(base + kGroupArrive) = 0u;
        *reinterpret_cast<uint32_t*>(base + kGroupState) = 0u;
    }
    unsigned long long* words = reinterpret_cast<unsigned long long*>(base + kGroupXw);
    constexpr int64_t nwords = (kGroupWordsEnd - kGroupXw) / (int64_t)sizeof(unsigned long long);
    for (int64_t k = threadIdx.x; k < nwords; k += kResetBlock) words[k] = 0ull;
}

// All-nodes schedule with row groups, for batches of few rows: S workgroups per node row
// (group g of group_of verifies row g of the node-major order, with its state at
// ws + g * kGroupStride).  The same chunks, slots and summation order as the row kernel,
// so the outcomes are identical; member 0 (or the member that claimed the row) writes
// them.
template <typename In, int VEC, int UNR, int MODE>
__global__ void __launch_bounds__(kPathBlock) __attribute__((amdgpu_waves_per_eu(2)))
rs_rowgroup_kernel(const KParams P, const GroupArgs ga) {
    __shared__ Smem sm;
    const int32_t S = ga.S;
    int32_t g, member;
    if (!group_of(ga, g, member)) return;
    int64_t row;
    int32_t b, n;
    if (P.flat) {
        row = g;
        b = g;
        n = 0;
    } else {
        n = g / P.B;
        b = g - n * P.B;
        row = (int64_t)b * P.N + n;
    }
    char* base = ga.ws + (int64_t)g * kGroupStride;
    RowGroup grp{S, member, reinterpret_cast<unsigned long long*>(base + kGroupXw),
                 reinterpret_cast<unsigned long long*>(base + kGroupXm), 0u, ga.wait};
    bool lead = member == 0;
    const int form = form_group(sm, grp, base, ga.form_wait);
    if (form == 0) return;   // another member does this row alone
    if (form == 2) {         // this member does it alone: every slot, no exchanges
        grp.S = 1;
        grp.w = 0;
        lead = true;
    }
    verify_row<In, VEC, UNR, MODE, kPathBlock, true>(P, sm, row, b, n, [&](int32_t child, int32_t tok, int32_t st) {
        if (lead) write_outcome(P, row, child, tok, st);
    }, grp);
}

// ----------------------------------------------------------- walk kernel ----

// One wave per sequence.  The walk itself is sequential, so the wave's lanes first load
// the outcomes of 64 consecutive nodes at once (one round trip instead of one per step);
// the walk then reads them across lanes, and loads the next 64 when it moves past them
// (children have larger indices than their parents).  Lane 0 writes the outputs.
constexpr int kWalkBlock = 256;

// Where a walk ended: the number of accepted draft tokens, the sequence's status, the node
// it ended at, and that node's token (-1 if none).  status RS_SEQ_DEFERRED: the walk ended
// at a node whose draw was deferred.
struct WalkEnd {
    int32_t len, status, node;
};

// One wave walks sequence `base / N` over the node outcomes: from the root it follows
// accepted children, writing each accepted node's token to out[0..len), and writes the
// token the last node drew (or its bonus) to out[len].  Lane 0 writes; every lane returns
// the same result.  The outcomes of 64 consecutive nodes are loaded at once, one per lane,
// and read across lanes as the walk steps (a child's index is larger than its parent's,
// so a new window is loaded only when the walk passes the current one).  Node ov_node
// takes the outcome (ov_child, ov_tok, ov_status) instead of the stored one (-1: none).
__device__ __forceinline__ WalkEnd walk_wave(const int32_t* __restrict__ node_child, const int32_t* __restrict__ node_tok,
                             const int32_t* __restrict__ node_status, const int32_t* __restrict__ node_token,
                             int64_t base, int32_t N, int32_t max_depth, int32_t* __restrict__ out,
                             int32_t ov_node, int32_t ov_child, int32_t ov_tok, int32_t ov_status) {
    const int lane = threadIdx.x & 63;
    const int64_t W = (int64_t)max_depth + 1;
    int32_t wbase = 0, wc = -1, wt = -1, ws = RS_SEQ_OK, wk = -1;
    auto window = [&](int32_t nb) {
        wbase = nb;
        const int32_t m = nb + lane;
        const bool in = m < N;
        wc = in ? node_child[base + m] : -1;
        wt = in ? node_tok[base + m] : -1;
        ws = in ? node_status[base + m] : RS_SEQ_OK;
        wk = in ? node_token[base + m] : -1;
        if (m == ov_node) {
            wc = ov_child;
            wt = ov_tok;
            ws = ov_status;
        }
    };
    window(0);
    if (lane == 0)
        for (int64_t i = 0; i < W; ++i) out[i] = -1;
    int32_t n = 0, len = 0, status = RS_SEQ_OK;
    for (int32_t steps = 0; steps <= N; ++steps) {
        if (n - wbase >= 64) window(n);
        const int k = n - wbase;
        const int32_t st = __builtin_amdgcn_readlane(ws, k);
        if (st != RS_SEQ_OK) {
            status = st;
            break;
        }
        const int32_t c = __builtin_amdgcn_readlane(wc, k);
        if (c >= 0) {
            if (c <= n || c >= N) {
                status = RS_SEQ_BAD_TREE;
                break;
            }
            if (len >= max_depth) {
                status = RS_SEQ_DEPTH_EXCEEDED;
                break;
            }
            if (c - wbase >= 64) window(c);
            const int32_t tk = __builtin_amdgcn_readlane(wk, c - wbase);
            if (lane == 0) out[len] = tk;
            ++len;
            n = c;
            continue;
        }
        const int32_t t = __builtin_amdgcn_readlane(wt, k);
        if (t >= 0 && lane == 0) out[len] = t;
        break;
    }
    return WalkEnd{len, status, n};
}

// The sequence's outputs once its walk has ended: on a fault every token and the length
// are -1.  Lane 0 writes.
__device__ __forceinline__ void walk_finish(const WalkEnd we, int64_t W, int32_t* __restrict__ out, int32_t b,
                            int32_t* __restrict__ out_len, int32_t* __restrict__ out_status) {
    if ((threadIdx.x & 63) != 0) return;
    int32_t len = we.len;
    if (we.status != RS_SEQ_OK) {
        for (int64_t i = 0; i < W; ++i) out[i] = -1;
        len = -1;
    }
    out_len[b] = len;
    if (out_status) out_status[b] = we.status;
}

// The walk of the all-nodes schedule: one wave per sequence.  It is latency-bound: every
// tree here fits one window of 64 nodes, so a sequence costs one round trip to memory.
__global__ void __launch_bounds__(kWalkBlock) rs_walk_kernel(const int32_t* __restrict__ node_child,
                                                             const int32_t* __restrict__ node_tok,
                                                             const int32_t* __restrict__ node_status,
                                                             const int32_t* __restrict__ node_token, int32_t B,
                                                             int32_t N, int32_t max_depth,
                                                             int32_t* __restrict__ out_tokens,
                                                             int32_t* __restrict__ out_len,
                                                             int32_t* __restrict__ out_status) {
    const int32_t b = (int32_t)(blockIdx.x * (kWalkBlock / 64) + (threadIdx.x >> 6));
    if (b >= B) return;   // the whole wave
    const int64_t W = (int64_t)max_depth + 1;
    int32_t* out = out_tokens + (int64_t)b * W;
    const WalkEnd we = walk_wave(node_child, node_tok, node_status, node_token, (int64_t)b * N, N, max_depth,
                                 out, -1, -1, -1, RS_SEQ_OK);
    walk_finish(we, W, out, b, out_len, out_status);
}

// The all-nodes schedule with deferred draws, first launch: every node row's tests, with
// the draws of single-candidate rejections and leaves deferred (same grid as the row
// kernel).
template <typename In, int VEC, int UNR, int MODE>
__global__ void __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(4))) rs_decide_kernel(const KParams P) {
    __shared__ Smem sm;
    const int32_t g = blockIdx.x;
    const int32_t n = g / P.B;
    const int32_t b = g - n * P.B;
    const int64_t row = (int64_t)b * P.N + n;
    RowGroup solo{1, 0, nullptr, nullptr, 0u, kGroupWaitTicks};
    verify_row<In, VEC, UNR, MODE, kBlock, false, false, kSchedDecide>(
        P, sm, row, b, n, [&](int32_t child, int32_t tok, int32_t st) { write_outcome(P, row, child, tok, st); },
        solo);
}

// Second launch: one workgroup per sequence walks the decided outcomes; where the walk
// ends at a row whose draw was deferred, the workgroup takes that row up again (its slot
// totals from the first launch, then its rejection pass and its draw, or the bonus draw
// of a leaf: pass 1, then the draw), records the node's outcome and finishes the walk
// with it.  Its workgroups are few (one per sequence), each streaming a row alone, so
// they take 12 waves (1.5 times the row kernel's loads in flight) and up to 168
// registers per lane: the row's code for a leaf, a single-candidate rejection and a row
// of several candidates is all in this kernel.
constexpr int kFinishBlock = 768;

template <typename In, int VEC, int UNR, int MODE>
__global__ void __launch_bounds__(kFinishBlock) __attribute__((amdgpu_waves_per_eu(2)))
rs_finish_kernel(const KParams P, int32_t max_depth, int32_t* __restrict__ out_tokens,
                 int32_t* __restrict__ out_len, int32_t* __restrict__ out_status) {
    constexpr int kBlock = kFinishBlock;
    __shared__ Smem sm;
    __shared__ int32_t s_node;
    const int32_t b = blockIdx.x;
    const int64_t W = (int64_t)max_depth + 1;
    int32_t* out = out_tokens + (int64_t)b * W;
    const int64_t base = (int64_t)b * P.N;
    WalkEnd we{0, RS_SEQ_OK, -1};
    if (threadIdx.x < 64) {
        we = walk_wave(P.node_child, P.node_tok, P.node_status, P.node_token, base, P.N, max_depth, out, -1, -1,
                       -1, RS_SEQ_OK);
        if (threadIdx.x == 0) s_node = we.status == RS_SEQ_DEFERRED ? we.node : -1;
    }
    __syncthreads();
    const int32_t n = s_node;
    if (n < 0) {
        if (threadIdx.x < 64) walk_finish(we, W, out, b, out_len, out_status);
        return;
    }
    const int64_t row = base + n;
    RowGroup solo{1, 0, nullptr, nullptr, 0u, kGroupWaitTicks};
    verify_row<In, VEC, UNR, MODE, kBlock, false, false, kSchedResume>(
        P, sm, row, b, n,
        [&](int32_t child, int32_t tok, int32_t st) {
            write_outcome(P, row, child, tok, st);
            sm.res_child = child;
            sm.res_tok = tok;
            sm.res_status = st;
        },
        solo);
    __syncthreads();
    if (threadIdx.x < 64) {
        const int32_t os = __builtin_amdgcn_readfirstlane(sm.res_status);
        int32_t oc = __builtin_amdgcn_readfirstlane(sm.res_child);
        int32_t ot = __builtin_amdgcn_readfirstlane(sm.res_tok);
        if (os != RS_SEQ_OK) oc = ot = -1;
        if (oc < 0) {
            // the walk ends here: the row's token (or its fault) completes the first walk
            if (os == RS_SEQ_OK && ot >= 0 && threadIdx.x == 0) out[we.len] = ot;
            we.status = os;
        } else {
            // (a resumed row repeats the test that deferred it, so this does not happen)
            we = walk_wave(P.node_child, P.node_tok, P.node_status, P.node_token, base, P.N, max_depth, out, n,
                           oc, ot, os);
        }
        walk_finish(we, W, out, b, out_len, out_status);
    }
}

}  // namespace

// ================================================================ host ABI ====

namespace {


// compute units of the current device (queried once per device)
// Workgroups of kPathBlock threads of kernel K that one CU holds at once, per device
// (cached: the answer depends only on the kernel's resources); 0 if the query fails.
template <auto K>
int resident_per_cu() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = -1;
    if (dev >= 0) {
        const int n = cache[dev].load(std::memory_order_relaxed);
        if (n > 0) return n;
    }
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(K), kPathBlock, 0) !=
        hipSuccess)
        per_cu = 0;
    if (dev >= 0 && per_cu > 0) cache[dev].store(per_cu, std::memory_order_relaxed);
    return per_cu;
}

int cu_count() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int n = cache[dev].load(std::memory_order_relaxed);
    if (n <= 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        cache[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

// Outputs of the path schedule (NULL: all-nodes schedule).
// time limits of row-group exchanges and formation for the next launches (a testing hook
// sets them)
std::atomic<uint64_t> g_group_wait{kGroupWaitTicks};
std::atomic<uint64_t> g_form_wait{kFormWaitTicks};

struct PathOut {
    int32_t max_depth;
    int32_t* out_tokens;
    int32_t* out_len;
    int32_t* out_status;
    int32_t group;       // members per sequence: 0 automatic, 1 one workgroup, >= 2 that many
    char* ws;            // row-group workspace (kGroupStride bytes per sequence) or null
    int dry_run;         // only resolve the group size
    int32_t used_group;  // out: members per sequence
    int unsupported;     // out: the requested group size cannot run on this device
};

// chunks of 64 * VEC * UNR elements, grouped into at most kMaxSlots slots of G chunks
template <int VEC, int UNR>
void set_slots(KParams& P) {
    constexpr int64_t CHUNK = 64 * VEC * UNR;
    const int64_t nch = ((int64_t)P.V + CHUNK - 1) / CHUNK;
    const int64_t G = (nch + kMaxSlots - 1) / kMaxSlots;
    P.G = (int32_t)G;
    P.nslots = (int32_t)((nch + G - 1) / G);
}

template <typename In, int VEC, int UNR, int MODE>
hipError_t launch_row_kernel(KParams P, int64_t nrows, hipStream_t s) {
    set_slots<VEC, UNR>(P);
    hipLaunchKernelGGL((rs_row_kernel<In, VEC, UNR, MODE>), dim3((unsigned)nrows), dim3(kBlock), 0, s, P);
    return hipGetLastError();
}

// Members per sequence: at most as many workgroups as the device holds at once (a group
// whose members do not all start in time is done by one of them alone), and each member
// keeps at least one slot (one per wave when chosen automatically).
template <typename In, int VEC, int UNR, int MODE>
int32_t resolve_group(const KParams& P, const PathOut* path) {
    if (path->group == 1 || (path->group == 0 && !path->ws)) return 1;
    if (!path->ws) return -1;
    const int64_t cap = (int64_t)resident_per_cu<rs_path_kernel<In, VEC, UNR, MODE>>() * cu_count();
    int64_t smax = (int64_t)kMaxGroup;
    if (cap / P.B < smax) smax = cap / P.B;
    if (path->group == 0) {
        // measured: with the tagged exchange, members of 4 slots still gain
        if (P.nslots / kPathAutoSlots < smax) smax = P.nslots / kPathAutoSlots;
        return smax >= 2 ? (int32_t)smax : 1;
    }
    if (P.nslots < smax) smax = P.nslots;
    return path->group <= smax ? path->group : -1;
}

template <typename In, int VEC, int UNR, int MODE>
hipError_t launch_path_kernel(KParams P, PathOut* path, hipStream_t s) {
    set_slots<VEC, UNR>(P);
    const int32_t S = resolve_group<In, VEC, UNR, MODE>(P, path);
    path->used_group = S;
    if (S < 1) {
        path->unsupported = 1;
        return hipErrorInvalidConfiguration;
    }
    if (path->dry_run) return hipSuccess;
    // The residual cache shortens the long walks, which set the step's time when the
    // launch leaves CUs free.  With more workgroups than CUs the step is bound by the
    // device's bandwidth instead, and the cache's extra traffic costs more than it saves
    // (measured on 1024 serving trees: 0.53 ms without, 0.58 ms with).
    if ((int64_t)P.B * S > (int64_t)cu_count()) P.rcache = nullptr;
    if (S == 1) {
        hipLaunchKernelGGL((rs_path_kernel<In, VEC, UNR, MODE>), dim3((unsigned)P.B), dim3(kPathBlock), 0, s,
                           P, path->max_depth, path->out_tokens, path->out_len, path->out_status,
                           GroupArgs{1, nullptr, kGroupWaitTicks, kFormWaitTicks, P.B, 0});
        return hipGetLastError();
    }
    // a row group per sequence: counters zeroed, then the members (which form their
    // groups themselves)
    hipLaunchKernelGGL(rs_group_reset, dim3((unsigned)P.B), dim3(kResetBlock), 0, s, path->ws, P.B);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    KParams kp = P;
    int32_t md = path->max_depth;
    int32_t* ot = path->out_tokens;
    int32_t* ol = path->out_len;
    int32_t* os = path->out_status;
    const bool xcd = S <= kXcdMaxMembers && P.B >= kXcdMinGroups;
    const GroupArgs ga{S, path->ws, g_group_wait.load(std::memory_order_relaxed),
                       g_form_wait.load(std::memory_order_relaxed), P.B, xcd ? 1 : 0};
    const int64_t groups = xcd ? ((int64_t)P.B + kXcds - 1) / kXcds * kXcds : (int64_t)P.B;
    hipLaunchKernelGGL((rs_path_kernel<In, VEC, UNR, MODE>), dim3((unsigned)(groups * S)), dim3(kPathBlock), 0, s,
                       kp, md, ot, ol, os, ga);
    return hipGetLastError();
}

// Row groups of the all-nodes schedule: the resolved size (1: the row kernel itself, no
// workspace used), -1 when the requested size cannot run.
struct RowGroupLaunch {
    int32_t group;       // members per row: 0 automatic, 1 one workgroup, >= 2 that many
    char* ws;            // nrows * kGroupStride bytes or null
    int dry_run;
    int32_t used_group;  // out
    int unsupported;     // out
};

template <typename In, int VEC, int UNR, int MODE>
hipError_t launch_rowgroups(KParams P, int64_t nrows, RowGroupLaunch* rg, hipStream_t s) {
    set_slots<VEC, UNR>(P);
    int32_t S = 1;
    if (rg->group >= 2 || (rg->group == 0 && rg->ws)) {
        const int64_t cap = (int64_t)resident_per_cu<rs_rowgroup_kernel<In, VEC, UNR, MODE>>() * cu_count();
        int64_t smax = (int64_t)kMaxGroup;
        if (cap / nrows < smax) smax = cap / nrows;
        if (rg->group == 0) {
            // measured: beyond one workgroup per CU, eight members per row or below 40 KiB
            // of a row per member, and for rows under 160 KiB, the exchanges cost more than
            // the split passes save
            if (kAutoRowGroup < smax) smax = kAutoRowGroup;
            const int64_t row_bytes = (int64_t)P.V * (int64_t)sizeof(In);
            const int64_t by_bytes = row_bytes < kAutoSplitBytes ? 1 : row_bytes / kAutoRowBytes;
            if (by_bytes < smax) smax = by_bytes;
            if ((int64_t)cu_count() / nrows < smax) smax = (int64_t)cu_count() / nrows;
            if (P.nslots / (kPathBlock / 64) < smax) smax = P.nslots / (kPathBlock / 64);
            S = smax >= 2 ? (int32_t)smax : 1;
        } else {
            if (P.nslots < smax) smax = P.nslots;
            S = (rg->group <= smax && rg->ws) ? rg->group : -1;
        }
    }
    rg->used_group = S;
    if (S < 1) {
        rg->unsupported = 1;
        return hipErrorInvalidConfiguration;
    }
    if (rg->dry_run) return hipSuccess;
    if (S == 1) {
        hipLaunchKernelGGL((rs_row_kernel<In, VEC, UNR, MODE>), dim3((unsigned)nrows), dim3(kBlock), 0, s, P);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(rs_group_reset, dim3((unsigned)nrows), dim3(kResetBlock), 0, s, rg->ws, (int32_t)nrows);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    KParams kp = P;
    const bool xcd = S <= kXcdMaxMembers && nrows >= kXcdMinGroups;
    const GroupArgs ga{S, rg->ws, g_group_wait.load(std::memory_order_relaxed),
                       g_form_wait.load(std::memory_order_relaxed), (int32_t)nrows, xcd ? 1 : 0};
    const int64_t groups = xcd ? (nrows + kXcds - 1) / kXcds * kXcds : nrows;
    hipLaunchKernelGGL((rs_rowgroup_kernel<In, VEC, UNR, MODE>), dim3((unsigned)(groups * S)), dim3(kPathBlock), 0,
                       s, kp, ga);
    return hipGetLastError();
}

template <int MODE>
hipError_t launch_rowgroups_m(const KParams& P, int dtype, bool vec, int64_t nrows, RowGroupLaunch* rg,
                              hipStream_t s) {
    if (dtype == RS_BF16)
        return vec ? launch_rowgroups<uint16_t, 8, kUnr16, MODE>(P, nrows, rg, s)
                   : launch_rowgroups<uint16_t, 1, 4, MODE>(P, nrows, rg, s);
    return vec ? launch_rowgroups<float, 4, kUnr32, MODE>(P, nrows, rg, s)
               : launch_rowgroups<float, 1, 4, MODE>(P, nrows, rg, s);
}

template <int MODE>
hipError_t launch_rows_m(const KParams& P, int dtype, bool vec, int64_t nrows, PathOut* path,
                         hipStream_t s) {
    if (path) {
        if (dtype == RS_BF16)
            return vec ? launch_path_kernel<uint16_t, 8, kUnr16, MODE>(P, path, s)
                       : launch_path_kernel<uint16_t, 1, 4, MODE>(P, path, s);
        return vec ? launch_path_kernel<float, 4, kUnr32, MODE>(P, path, s)
                   : launch_path_kernel<float, 1, 4, MODE>(P, path, s);
    }
    if (dtype == RS_BF16) {
        return vec ? launch_row_kernel<uint16_t, 8, kUnr16, MODE>(P, nrows, s)
                   : launch_row_kernel<uint16_t, 1, 4, MODE>(P, nrows, s);
    }
    return vec ? launch_row_kernel<float, 4, kUnr32, MODE>(P, nrows, s)
               : launch_row_kernel<float, 1, 4, MODE>(P, nrows, s);
}
hipError_t launch_rows(const KParams& P, const rs_params* prm, bool vec, int64_t nrows, hipStream_t s,
                       PathOut* path = nullptr) {
    if (prm->mode == RS_MODE_SPECINFER)
        return launch_rows_m<RS_MODE_SPECINFER>(P, prm->logits_dtype, vec, nrows, path, s);
    return launch_rows_m<RS_MODE_RESISPEC>(P, prm->logits_dtype, vec, nrows, path, s);
}

bool vector_ok(const void* t, const void* d, int64_t V, int dtype) {
    const int64_t esz = dtype == RS_BF16 ? 2 : 4;
    return ((V * esz) % 16 == 0) && aligned16(t) && aligned16(d);
}

KParams base_params(const void* t, const void* d, int64_t V, const rs_params* prm) {
    KParams P{};
    P.tgt = t;
    P.dft = d;
    P.V = (int32_t)V;
    P.T = prm->temperature;
    split_c2(prm->temperature, &P.c2h, &P.c2l);
    P.worep = prm->without_replacement ? 1 : 0;
    P.bonus = prm->bonus ? 1 : 0;
    return P;
}

size_t node_arrays_bytes(int64_t rows) {
    const size_t one = ((size_t)rows * sizeof(int32_t) + 255) & ~(size_t)255;
    return 3 * one;
}

hipError_t launch_walk(const int32_t* node_child, const int32_t* node_tok,
                       const int32_t* node_status, const int32_t* node_token, int32_t B, int32_t N,
                       int32_t max_depth, int32_t* out_tokens, int32_t* out_len,
                       int32_t* out_status, hipStream_t s) {
    constexpr int per_block = kWalkBlock / 64;   // one wave per sequence
    hipLaunchKernelGGL(rs_walk_kernel, dim3((unsigned)((B + per_block - 1) / per_block)),
                       dim3(kWalkBlock), 0, s, node_child, node_tok, node_status, node_token, B, N,
                       max_depth, out_tokens, out_len, out_status);
    return hipGetLastError();
}

// Deferred draws: the decide kernel over every node row, or the finish kernel over every
// sequence (finish = true).
template <typename In, int VEC, int UNR, int MODE>
hipError_t launch_deferred(KParams P, bool finish, int32_t max_depth, int32_t* out_tokens, int32_t* out_len,
                           int32_t* out_status, hipStream_t s) {
    set_slots<VEC, UNR>(P);
    if (finish)
        hipLaunchKernelGGL((rs_finish_kernel<In, VEC, UNR, MODE>), dim3((unsigned)P.B), dim3(kFinishBlock), 0, s, P,
                           max_depth, out_tokens, out_len, out_status);
    else
        hipLaunchKernelGGL((rs_decide_kernel<In, VEC, UNR, MODE>), dim3((unsigned)((int64_t)P.B * P.N)),
                           dim3(kBlock), 0, s, P);
    return hipGetLastError();
}

template <int MODE>
hipError_t launch_deferred_m(const KParams& P, int dtype, bool vec, bool finish, int32_t max_depth,
                             int32_t* out_tokens, int32_t* out_len, int32_t* out_status, hipStream_t s) {
    if (dtype == RS_BF16)
        return vec ? launch_deferred<uint16_t, 8, kUnr16, MODE>(P, finish, max_depth, out_tokens, out_len,
                                                                out_status, s)
                   : launch_deferred<uint16_t, 1, 4, MODE>(P, finish, max_depth, out_tokens, out_len, out_status, s);
    return vec ? launch_deferred<float, 4, kUnr32, MODE>(P, finish, max_depth, out_tokens, out_len, out_status, s)
               : launch_deferred<float, 1, 4, MODE>(P, finish, max_depth, out_tokens, out_len, out_status, s);
}

hipError_t launch_deferred_stage(const KParams& P, const rs_params* prm, bool vec, bool finish, int32_t max_depth,
                                 int32_t* out_tokens, int32_t* out_len, int32_t* out_status, hipStream_t s) {
    if (prm->mode == RS_MODE_SPECINFER)
        return launch_deferred_m<RS_MODE_SPECINFER>(P, prm->logits_dtype, vec, finish, max_depth, out_tokens,
                                                    out_len, out_status, s);
    return launch_deferred_m<RS_MODE_RESISPEC>(P, prm->logits_dtype, vec, finish, max_depth, out_tokens, out_len,
                                               out_status, s);
}

// bytes of the deferred schedule's workspace: the node outcome arrays, then the slot
// totals of every row
size_t deferred_bytes(int64_t rows) {
    return node_arrays_bytes(rows) + (size_t)rows * (size_t)kStateDoubles * sizeof(double);
}

KParams tree_params(const void* target_logits, const void* draft_logits, const int32_t* node_token,
                    const int32_t* parent, const float* u_accept, const float* u_resample,
                    int32_t B, int32_t N, int32_t V, const rs_params* prm, int32_t* node_child,
                    int32_t* node_tok, int32_t* node_status, float* residual_out) {
    KParams P = base_params(target_logits, draft_logits, V, prm);
    P.flat = 0;
    P.node_token = node_token;
    P.parent = parent;
    P.ua = u_accept;
    P.ur = u_resample;
    P.node_child = node_child;
    P.node_tok = node_tok;
    P.node_status = node_status;
    P.residual_out = residual_out;
    P.B = B;
    P.N = N;
    return P;
}

rs_status tree_impl(const void* target_logits, const void* draft_logits, const int32_t* node_token,
                    const int32_t* parent, const float* u_accept, const float* u_resample, int32_t B,
                    int32_t N, int32_t V, int32_t max_depth, const rs_params* prm, int32_t* out_tokens,
                    int32_t* out_accepted_len, int32_t* out_status, int32_t* node_child,
                    int32_t* node_tok, int32_t* node_status, float* residual_out, hipStream_t s) {
    const KParams P = tree_params(target_logits, draft_logits, node_token, parent, u_accept,
                                  u_resample, B, N, V, prm, node_child, node_tok, node_status,
                                  residual_out);
    const bool vec = vector_ok(target_logits, draft_logits, V, prm->logits_dtype);
    if (launch_rows(P, prm, vec, (int64_t)B * N, s) != hipSuccess) return RS_ERR_HIP;
    return launch_walk(node_child, node_tok, node_status, node_token, B, N, max_depth, out_tokens,
                       out_accepted_len, out_status, s) == hipSuccess ? RS_OK : RS_ERR_HIP;
}

int32_t* ws_array(void* workspace, int64_t rows, int which) {
    const size_t one = node_arrays_bytes(rows) / 3;
    return reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + which * one);
}

rs_status check_tree_args(const void* target_logits, const void* draft_logits,
                          const int32_t* node_token, const int32_t* parent, const float* u_accept,
                          const float* u_resample, int32_t B, int32_t N, int32_t V,
                          int32_t max_depth, const rs_params* prm, const int32_t* out_tokens,
                          const int32_t* out_accepted_len) {
    const rs_status ps = check_params(prm);
    if (ps != RS_OK) return ps;
    if (B < 0 || N <= 0 || V <= 0 || max_depth < 0) return RS_ERR_INVALID_ARG;
    if (V > RS_MAX_VOCAB) return RS_ERR_UNSUPPORTED;
    if ((int64_t)B * N > 0x7fffffffLL) return RS_ERR_UNSUPPORTED;
    if (B == 0) return RS_OK;
    if (!target_logits || !draft_logits || !node_token || !parent || !u_accept || !u_resample ||
        !out_tokens || !out_accepted_len)
        return RS_ERR_INVALID_ARG;
    return RS_OK;
}

}  // namespace

// Scratch of the entry point that allocates nothing (resispec_verify_tree_noalloc): the
// per-node outcome arrays of RS_NOALLOC_MAX_ROWS node rows, laid out as the caller
// workspace of resispec_verify_tree.  Every GPU the library runs on holds one copy until
// the process ends; its device address is looked up once per device (in host code the
// array's name is not a device address).
constexpr int64_t kNoAllocRows = RS_NOALLOC_MAX_ROWS;
constexpr size_t kNoAllocBytes = 3 * (((size_t)kNoAllocRows * sizeof(int32_t) + 255) & ~(size_t)255);
__device__ __align__(256) char scratch[kNoAllocBytes];

namespace {

std::mutex g_scratch_mu;
void* g_scratch_ptr[64];   // per device, null until looked up

// The current device's address of `scratch` (null if the lookup fails).
void* scratch_ptr() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

int32_t resispec_abi_version(void) { return RESISPEC_ABI_VERSION; }

const char* resispec_status_string(int32_t status) {
    switch (status) {
        case RS_OK: return "RS_OK";
        case RS_ERR_INVALID_ARG: return "RS_ERR_INVALID_ARG: invalid argument";
        case RS_ERR_WORKSPACE: return "RS_ERR_WORKSPACE: workspace missing or too small";
        case RS_ERR_UNSUPPORTED: return "RS_ERR_UNSUPPORTED: size beyond the supported limits";
        case RS_ERR_HIP: return "RS_ERR_HIP: HIP launch error";
        default: return "unknown rs_status";
    }
}

size_t resispec_workspace_bytes(int32_t B, int32_t N) {
    if (B <= 0 || N <= 0) return 0;
    return node_arrays_bytes((int64_t)B * N);
}

rs_status resispec_verify(const void* target_logits, const void* draft_logits,
                          const int32_t* cand_ids, const float* u_accept,
                          const float* u_resample, int32_t B, int32_t V, int32_t k,
                          const rs_params* prm, int32_t* out_token, int32_t* out_accepted_len,
                          int32_t* out_status, void* stream) {
    const rs_status ps = check_params(prm);
    if (ps != RS_OK) return ps;
    if (B < 0 || V <= 0 || k < 0) return RS_ERR_INVALID_ARG;
    if (V > RS_MAX_VOCAB || k > RS_MAX_CANDIDATES) return RS_ERR_UNSUPPORTED;
    if (B == 0) return RS_OK;
    if (!target_logits || !u_resample || !out_token || !out_accepted_len) return RS_ERR_INVALID_ARG;
    if (k > 0 && (!draft_logits || !cand_ids || !u_accept)) return RS_ERR_INVALID_ARG;
    const void* draft = draft_logits ? draft_logits : target_logits;   // k = 0 never reads it
    KParams P = base_params(target_logits, draft, V, prm);
    P.flat = 1;
    P.bonus = 1;
    P.cand_ids = cand_ids;
    P.ua_flat = u_accept;
    P.ur_flat = u_resample;
    P.k = k;
    P.out_token = out_token;
    P.out_len = out_accepted_len;
    P.out_status = out_status;
    P.B = B;
    P.N = 1;
    const bool vec = vector_ok(target_logits, draft, V, prm->logits_dtype);
    return launch_rows(P, prm, vec, B, (hipStream_t)stream) == hipSuccess ? RS_OK : RS_ERR_HIP;
}

rs_status resispec_verify_tree(const void* target_logits, const void* draft_logits,
                               const int32_t* node_token, const int32_t* parent,
                               const float* u_accept, const float* u_resample, int32_t B,
                               int32_t N, int32_t V, int32_t max_depth, const rs_params* prm,
                               int32_t* out_tokens, int32_t* out_accepted_len, int32_t* out_status,
                               void* workspace, size_t workspace_bytes, void* stream) {
    const rs_status as = check_tree_args(target_logits, draft_logits, node_token, parent, u_accept,
                                         u_resample, B, N, V, max_depth, prm, out_tokens,
                                         out_accepted_len);
    if (as != RS_OK || B == 0) return as;
    if (!workspace || workspace_bytes < resispec_workspace_bytes(B, N) || !aligned16(workspace))
        return RS_ERR_WORKSPACE;
    const int64_t rows = (int64_t)B * N;
    return tree_impl(target_logits, draft_logits, node_token, parent, u_accept, u_resample, B, N, V,
                     max_depth, prm, out_tokens, out_accepted_len, out_status,
                     ws_array(workspace, rows, 0), ws_array(workspace, rows, 1),
                     ws_array(workspace, rows, 2), nullptr, (hipStream_t)stream);
}

rs_status resispec_verify_tree_noalloc(const void* target_logits, const void* draft_logits,
                                       const int32_t* node_token, const int32_t* parent,
                                       const float* u_accept, const float* u_resample,
                                       int32_t B, int32_t N, int32_t V, int32_t max_depth,
                                       const rs_params* prm, int32_t* out_tokens,
                                       int32_t* out_accepted_len, int32_t* out_status,
                                       void* stream) {
    const rs_status as = check_tree_args(target_logits, draft_logits, node_token, parent, u_accept,
                                         u_resample, B, N, V, max_depth, prm, out_tokens,
                                         out_accepted_len);
    if (as != RS_OK || B == 0) return as;
    const int64_t rows = (int64_t)B * N;
    if (rows > kNoAllocRows) return RS_ERR_UNSUPPORTED;
    void* ws = scratch_ptr();
    if (!ws) return RS_ERR_HIP;
    // the node arrays of `rows` rows fit the scratch laid out for kNoAllocRows rows; the
    // row kernel writes every row's outcome before the walk reads it, so nothing needs
    // clearing between calls
    return tree_impl(target_logits, draft_logits, node_token, parent, u_accept, u_resample, B, N, V,
                     max_depth, prm, out_tokens, out_accepted_len, out_status,
                     ws_array(ws, rows, 0), ws_array(ws, rows, 1), ws_array(ws, rows, 2), nullptr,
                     (hipStream_t)stream);
}

size_t resispec_tree_group_workspace_bytes(int32_t B, int32_t N) {
    if (B <= 0 || N <= 0) return 0;
    const int64_t rows = (int64_t)B * N;
    return node_arrays_bytes(rows) + (size_t)rows * (size_t)kGroupStride;
}

rs_status resispec_verify_tree_group(const void* target_logits, const void* draft_logits,
                                     const int32_t* node_token, const int32_t* parent,
                                     const float* u_accept, const float* u_resample, int32_t B,
                                     int32_t N, int32_t V, int32_t max_depth, const rs_params* prm,
                                     int32_t* out_tokens, int32_t* out_accepted_len,
                                     int32_t* out_status, int32_t group_size, void* workspace,
                                     size_t workspace_bytes, void* stream) {
    const rs_status as = check_tree_args(target_logits, draft_logits, node_token, parent, u_accept,
                                         u_resample, B, N, V, max_depth, prm, out_tokens,
                                         out_accepted_len);
    if (as != RS_OK) return as;
    if (group_size < 0 || group_size > kMaxGroup) return RS_ERR_INVALID_ARG;
    if (B == 0) return RS_OK;
    if (!workspace || workspace_bytes < resispec_tree_group_workspace_bytes(B, N) || !aligned16(workspace))
        return RS_ERR_WORKSPACE;
    const int64_t rows = (int64_t)B * N;
    int32_t* nc = ws_array(workspace, rows, 0);
    int32_t* nt = ws_array(workspace, rows, 1);
    int32_t* ns = ws_array(workspace, rows, 2);
    const KParams P = tree_params(target_logits, draft_logits, node_token, parent, u_accept,
                                  u_resample, B, N, V, prm, nc, nt, ns, nullptr);
    const bool vec = vector_ok(target_logits, draft_logits, V, prm->logits_dtype);
    RowGroupLaunch rg{group_size, static_cast<char*>(workspace) + node_arrays_bytes(rows), 0, 1, 0};
    const hipStream_t s = (hipStream_t)stream;
    const hipError_t e = prm->mode == RS_MODE_SPECINFER
                             ? launch_rowgroups_m<RS_MODE_SPECINFER>(P, prm->logits_dtype, vec, rows, &rg, s)
                             : launch_rowgroups_m<RS_MODE_RESISPEC>(P, prm->logits_dtype, vec, rows, &rg, s);
    if (rg.unsupported) return RS_ERR_UNSUPPORTED;
    if (e != hipSuccess) return RS_ERR_HIP;
    return launch_walk(nc, nt, ns, node_token, B, N, max_depth, out_tokens, out_accepted_len,
                       out_status, s) == hipSuccess ? RS_OK : RS_ERR_HIP;
}

int32_t resispec_tree_group_size(int32_t B, int32_t N, int32_t V, const rs_params* prm) {
    if (B <= 0 || N <= 0 || V <= 0 || !prm || (prm->logits_dtype != RS_F32 && prm->logits_dtype != RS_BF16) ||
        (prm->mode != RS_MODE_RESISPEC && prm->mode != RS_MODE_SPECINFER))
        return -1;
    KParams P{};
    P.B = B;
    P.N = N;
    P.V = V;
    char probe = 0;   // any non-null workspace: the answer does not depend on it
    RowGroupLaunch rg{0, &probe, 1, 1, 0};
    const bool vec = (prm->logits_dtype == RS_BF16) ? (V % 8 == 0) : (V % 4 == 0);
    const int64_t rows = (int64_t)B * N;
    const hipError_t e = prm->mode == RS_MODE_SPECINFER
                             ? launch_rowgroups_m<RS_MODE_SPECINFER>(P, prm->logits_dtype, vec, rows, &rg, nullptr)
                             : launch_rowgroups_m<RS_MODE_RESISPEC>(P, prm->logits_dtype, vec, rows, &rg, nullptr);
    return e == hipSuccess ? rg.used_group : -1;
}

// Path workspace: one group state per sequence, then the residual cache (rc_stride(V)
// floats per sequence, starting on a 256-byte boundary: the residual R, then the draft
// masses Q, each V rounded up to a multiple of kRcPad).
static size_t path_states_bytes(int32_t B) { return ((size_t)B * (size_t)kGroupStride + 255) & ~(size_t)255; }
static int64_t rc_stride(int32_t V) { return 2 * (((int64_t)V + kRcPad - 1) / kRcPad * kRcPad); }

static rs_status verify_tree_path_impl(const void* target_logits, const void* draft_logits,
                                       const int32_t* node_token, const int32_t* parent,
                                       const float* u_accept, const float* u_resample, int32_t B,
                                       int32_t N, int32_t V, int32_t max_depth, const rs_params* prm,
                                       int32_t* out_tokens, int32_t* out_accepted_len,
                                       int32_t* out_status, int32_t group_size, void* workspace,
                                       size_t workspace_bytes, void* stream) {
    const rs_status as = check_tree_args(target_logits, draft_logits, node_token, parent, u_accept,
                                         u_resample, B, N, V, max_depth, prm, out_tokens,
                                         out_accepted_len);
    if (as != RS_OK) return as;
    if (group_size < 0 || group_size > kMaxGroup) return RS_ERR_INVALID_ARG;
    if (workspace && (workspace_bytes < resispec_path_workspace_bytes(B, V) || !aligned16(workspace)))
        return RS_ERR_WORKSPACE;
    if (group_size >= 2 && !workspace) return RS_ERR_WORKSPACE;
    if (B == 0) return RS_OK;
    KParams P = tree_params(target_logits, draft_logits, node_token, parent, u_accept,
                            u_resample, B, N, V, prm, nullptr, nullptr, nullptr, nullptr);
    if (workspace) {
        // the residual cache follows the group states
        P.rcache = reinterpret_cast<float*>(static_cast<char*>(workspace) + path_states_bytes(B));
        P.rc_stride = rc_stride(V);
    }
    const bool vec = vector_ok(target_logits, draft_logits, V, prm->logits_dtype);
    PathOut path{max_depth, out_tokens, out_accepted_len, out_status, group_size,
                 static_cast<char*>(workspace), 0, 1, 0};
    const hipError_t e = launch_rows(P, prm, vec, B, (hipStream_t)stream, &path);
    if (path.unsupported) return RS_ERR_UNSUPPORTED;
    return e == hipSuccess ? RS_OK : RS_ERR_HIP;
}

rs_status resispec_verify_tree_path(const void* target_logits, const void* draft_logits,
                                    const int32_t* node_token, const int32_t* parent,
                                    const float* u_accept, const float* u_resample, int32_t B,
                                    int32_t N, int32_t V, int32_t max_depth, const rs_params* prm,
                                    int32_t* out_tokens, int32_t* out_accepted_len,
                                    int32_t* out_status, void* stream) {
    return verify_tree_path_impl(target_logits, draft_logits, node_token, parent, u_accept,
                                 u_resample, B, N, V, max_depth, prm, out_tokens, out_accepted_len,
                                 out_status, 1, nullptr, 0, stream);
}

rs_status resispec_verify_tree_path_group(const void* target_logits, const void* draft_logits,
                                          const int32_t* node_token, const int32_t* parent,
                                          const float* u_accept, const float* u_resample,
                                          int32_t B, int32_t N, int32_t V, int32_t max_depth,
                                          const rs_params* prm, int32_t* out_tokens,
                                          int32_t* out_accepted_len, int32_t* out_status,
                                          int32_t group_size, void* workspace,
                                          size_t workspace_bytes, void* stream) {
    return verify_tree_path_impl(target_logits, draft_logits, node_token, parent, u_accept,
                                 u_resample, B, N, V, max_depth, prm, out_tokens, out_accepted_len,
                                 out_status, group_size, workspace, workspace_bytes, stream);
}

rs_status resispec_debug_set_group_waits(uint64_t barrier_ticks, uint64_t formation_ticks) {
    g_group_wait.store(barrier_ticks == UINT64_MAX ? kGroupWaitTicks : barrier_ticks, std::memory_order_relaxed);
    g_form_wait.store(formation_ticks == UINT64_MAX ? kFormWaitTicks : formation_ticks, std::memory_order_relaxed);
    return RS_OK;
}

size_t resispec_path_workspace_bytes(int32_t B, int32_t V) {
    if (B <= 0 || V <= 0 || V > RS_MAX_VOCAB) return 0;
    return path_states_bytes(B) + (size_t)B * (size_t)rc_stride(V) * sizeof(float);
}

int32_t resispec_path_group_size(int32_t B, int32_t V, const rs_params* prm) {
    if (B <= 0 || V <= 0 || !prm || (prm->logits_dtype != RS_F32 && prm->logits_dtype != RS_BF16) ||
        (prm->mode != RS_MODE_RESISPEC && prm->mode != RS_MODE_SPECINFER))
        return -1;
    KParams P{};
    P.B = B;
    P.V = V;
    char probe = 0;   // any non-null workspace: the answer does not depend on it
    PathOut path{0, nullptr, nullptr, nullptr, 0, &probe, 1, 1, 0};
    // 16-byte aligned rows take the vector kernels
    const bool vec = (prm->logits_dtype == RS_BF16) ? (V % 8 == 0) : (V % 4 == 0);
    if (launch_rows(P, prm, vec, B, nullptr, &path) != hipSuccess) return -1;
    return path.used_group;
}

rs_status resispec_verify_nodes(const void* target_logits, const void* draft_logits,
                                const int32_t* node_token, const int32_t* parent,
                                const float* u_accept, const float* u_resample, int32_t B,
                                int32_t N, int32_t V, const rs_params* prm, void* workspace,
                                size_t workspace_bytes, void* stream) {
    int32_t dummy = 0;   // output pointers are not used by this stage
    const rs_status as = check_tree_args(target_logits, draft_logits, node_token, parent, u_accept,
                                         u_resample, B, N, V, 0, prm, &dummy, &dummy);
    if (as != RS_OK || B == 0) return as;
    if (!workspace || workspace_bytes < resispec_workspace_bytes(B, N) || !aligned16(workspace))
        return RS_ERR_WORKSPACE;
    const int64_t rows = (int64_t)B * N;
    const KParams P = tree_params(target_logits, draft_logits, node_token, parent, u_accept,
                                  u_resample, B, N, V, prm, ws_array(workspace, rows, 0),
                                  ws_array(workspace, rows, 1), ws_array(workspace, rows, 2),
                                  nullptr);
    const bool vec = vector_ok(target_logits, draft_logits, V, prm->logits_dtype);
    return launch_rows(P, prm, vec, rows, (hipStream_t)stream) == hipSuccess ? RS_OK : RS_ERR_HIP;
}

rs_status resispec_walk(const int32_t* node_token, int32_t B, int32_t N, int32_t max_depth,
                        const void* workspace, size_t workspace_bytes, int32_t* out_tokens,
                        int32_t* out_accepted_len, int32_t* out_status, void* stream) {
    if (B < 0 || N <= 0 || max_depth < 0) return RS_ERR_INVALID_ARG;
    if ((int64_t)B * N > 0x7fffffffLL) return RS_ERR_UNSUPPORTED;
    if (B == 0) return RS_OK;
    if (!node_token || !out_tokens || !out_accepted_len) return RS_ERR_INVALID_ARG;
    if (!workspace || workspace_bytes < resispec_workspace_bytes(B, N) || !aligned16(workspace))
        return RS_ERR_WORKSPACE;
    const int64_t rows = (int64_t)B * N;
    void* ws = const_cast<void*>(workspace);
    return launch_walk(ws_array(ws, rows, 0), ws_array(ws, rows, 1), ws_array(ws, rows, 2),
                       node_token, B, N, max_depth, out_tokens, out_accepted_len, out_status,
                       (hipStream_t)stream) == hipSuccess ? RS_OK : RS_ERR_HIP;
}

rs_status resispec_node_outcomes(const void* workspace, size_t workspace_bytes, int32_t B,
                                 int32_t N, int32_t* node_child, int32_t* node_token_out,
                                 int32_t* node_status, void* stream) {
    if (B < 0 || N <= 0) return RS_ERR_INVALID_ARG;
    if ((int64_t)B * N > 0x7fffffffLL) return RS_ERR_UNSUPPORTED;
    if (B == 0) return RS_OK;
    if (!node_child || !node_token_out || !node_status) return RS_ERR_INVALID_ARG;
    if (!workspace || workspace_bytes < resispec_workspace_bytes(B, N) || !aligned16(workspace))
        return RS_ERR_WORKSPACE;
    const int64_t rows = (int64_t)B * N;
    void* ws = const_cast<void*>(workspace);
    int32_t* dst[3] = {node_child, node_token_out, node_status};
    for (int k = 0; k < 3; ++k)
        if (hipMemcpyAsync(dst[k], ws_array(ws, rows, k), (size_t)rows * sizeof(int32_t),
                           hipMemcpyDeviceToDevice, (hipStream_t)stream) != hipSuccess)
            return RS_ERR_HIP;
    return RS_OK;
}

rs_status resispec_verify_tree_debug(const void* target_logits, const void* draft_logits,
                                     const int32_t* node_token, const int32_t* parent,
                                     const float* u_accept, const float* u_resample, int32_t B,
                                     int32_t N, int32_t V, int32_t max_depth, const rs_params* prm,
                                     int32_t* out_tokens, int32_t* out_accepted_len,
                                     int32_t* out_status, void* workspace, size_t workspace_bytes,
                                     int32_t* node_child, int32_t* node_token_out,
                                     int32_t* node_status, float* residual_out, void* stream) {
    (void)workspace;
    (void)workspace_bytes;
    const rs_status as = check_tree_args(target_logits, draft_logits, node_token, parent, u_accept,
                                         u_resample, B, N, V, max_depth, prm, out_tokens,
                                         out_accepted_len);
    if (as != RS_OK || B == 0) return as;
    if (!node_child || !node_token_out || !node_status) return RS_ERR_INVALID_ARG;
    return tree_impl(target_logits, draft_logits, node_token, parent, u_accept, u_resample, B, N, V,
                     max_depth, prm, out_tokens, out_accepted_len, out_status, node_child,
                     node_token_out, node_status, residual_out, (hipStream_t)stream);
}

size_t resispec_deferred_workspace_bytes(int32_t B, int32_t N) {
    if (B <= 0 || N <= 0) return 0;
    return deferred_bytes((int64_t)B * N);
}

}  // extern "C"

namespace {

// One stage of the deferred schedule: the decide launch (finish = false) or the walk with
// the deferred draws (finish = true).
rs_status deferred_stage(const void* target_logits, const void* draft_logits, const int32_t* node_token,
                         const int32_t* parent, const float* u_accept, const float* u_resample, int32_t B,
                         int32_t N, int32_t V, int32_t max_depth, const rs_params* prm, int32_t* out_tokens,
                         int32_t* out_accepted_len, int32_t* out_status, void* workspace,
                         size_t workspace_bytes, bool finish, hipStream_t s) {
    const int64_t rows = (int64_t)B * N;
    KParams P = tree_params(target_logits, draft_logits, node_token, parent, u_accept, u_resample, B, N, V, prm,
                            ws_array(workspace, rows, 0), ws_array(workspace, rows, 1),
                            ws_array(workspace, rows, 2), nullptr);
    P.dstate = reinterpret_cast<double*>(static_cast<char*>(workspace) + node_arrays_bytes(rows));
    const bool vec = vector_ok(target_logits, draft_logits, V, prm->logits_dtype);
    return launch_deferred_stage(P, prm, vec, finish, max_depth, out_tokens, out_accepted_len, out_status, s) ==
                   hipSuccess
               ? RS_OK
               : RS_ERR_HIP;
}

bool deferred_ws_ok(const void* workspace, size_t workspace_bytes, int32_t B, int32_t N) {
    return workspace && aligned16(workspace) && workspace_bytes >= resispec_deferred_workspace_bytes(B, N);
}

}  // namespace

extern "C" {

rs_status resispec_decide_nodes(const void* target_logits, const void* draft_logits,
                                const int32_t* node_token, const int32_t* parent,
                                const float* u_accept, const float* u_resample, int32_t B,
                                int32_t N, int32_t V, const rs_params* prm, void* workspace,
                                size_t workspace_bytes, void* stream) {
    int32_t dummy = 0;   // output pointers are not used by this stage
    const rs_status as = check_tree_args(target_logits, draft_logits, node_token, parent, u_accept,
                                         u_resample, B, N, V, 0, prm, &dummy, &dummy);
    if (as != RS_OK || B == 0) return as;
    if (!deferred_ws_ok(workspace, workspace_bytes, B, N)) return RS_ERR_WORKSPACE;
    return deferred_stage(target_logits, draft_logits, node_token, parent, u_accept, u_resample, B, N, V, 0, prm,
                          nullptr, nullptr, nullptr, workspace, workspace_bytes, false, (hipStream_t)stream);
}

rs_status resispec_walk_draw(const void* target_logits, const void* draft_logits,
                             const int32_t* node_token, const int32_t* parent,
                             const float* u_accept, const float* u_resample, int32_t B,
                             int32_t N, int32_t V, int32_t max_depth, const rs_params* prm,
                             void* workspace, size_t workspace_bytes, int32_t* out_tokens,
                             int32_t* out_accepted_len, int32_t* out_status, void* stream) {
    const rs_status as = check_tree_args(target_logits, draft_logits, node_token, parent, u_accept,
                                         u_resample, B, N, V, max_depth, prm, out_tokens,
                                         out_accepted_len);
    if (as != RS_OK || B == 0) return as;
    if (!deferred_ws_ok(workspace, workspace_bytes, B, N)) return RS_ERR_WORKSPACE;
    return deferred_stage(target_logits, draft_logits, node_token, parent, u_accept, u_resample, B, N, V,
                          max_depth, prm, out_tokens, out_accepted_len, out_status, workspace, workspace_bytes,
                          true, (hipStream_t)stream);
}

rs_status resispec_verify_tree_deferred(const void* target_logits, const void* draft_logits,
                                        const int32_t* node_token, const int32_t* parent,
                                        const float* u_accept, const float* u_resample, int32_t B,
                                        int32_t N, int32_t V, int32_t max_depth, const rs_params* prm,
                                        int32_t* out_tokens, int32_t* out_accepted_len,
                                        int32_t* out_status, void* workspace, size_t workspace_bytes,
                                        void* stream) {
    const rs_status as = check_tree_args(target_logits, draft_logits, node_token, parent, u_accept,
                                         u_resample, B, N, V, max_depth, prm, out_tokens,
                                         out_accepted_len);
    if (as != RS_OK || B == 0) return as;
    if (!deferred_ws_ok(workspace, workspace_bytes, B, N)) return RS_ERR_WORKSPACE;
    const hipStream_t s = (hipStream_t)stream;
    const rs_status r = deferred_stage(target_logits, draft_logits, node_token, parent, u_accept, u_resample, B,
                                       N, V, max_depth, prm, out_tokens, out_accepted_len, out_status, workspace,
                                       workspace_bytes, false, s);
    if (r != RS_OK) return r;
    return deferred_stage(target_logits, draft_logits, node_token, parent, u_accept, u_resample, B, N, V,
                          max_depth, prm, out_tokens, out_accepted_len, out_status, workspace, workspace_bytes,
                          true, s);
}

rs_status resispec_validate_tree_host(const int32_t* parent, const int32_t* node_token, int32_t B,
                                      int32_t N, int32_t V, int64_t* first_bad) {
    if (first_bad) *first_bad = -1;
    if (B < 0 || N <= 0 || V <= 0) return RS_ERR_INVALID_ARG;
    if (B > 0 && (!parent || !node_token)) return RS_ERR_INVALID_ARG;
    for (int64_t b = 0; b < B; ++b) {
        const int32_t* par = parent + b * N;
        const int32_t* tok = node_token + b * N;
        for (int32_t n = 0; n < N; ++n) {
            const bool bad_parent = (n == 0) ? (par[0] != -1) : (par[n] < 0 || par[n] >= n);
            const bool bad_token = n > 0 && (tok[n] < 0 || tok[n] >= V);
            if (bad_parent || bad_token) {
                if (first_bad) *first_bad = b * N + n;
                return RS_ERR_INVALID_ARG;
            }
        }
        // children per node
        for (int32_t n = 0; n < N; ++n) {
            int32_t c = 0;
            for (int32_t m = n + 1; m < N; ++m) c += (par[m] == n);
            if (c > RS_MAX_CANDIDATES) {
                if (first_bad) *first_bad = b * N + n;
                return RS_ERR_INVALID_ARG;
            }
        }
    }
    return RS_OK;
}

}  // extern "C"
