// common.h -- constants and device helpers shared by the verification kernels
// (resispec.hip) and the draft-step kernel (draft.hip): vector loads of logits rows,
// the exponent evaluation, wavefront reductions, the workgroup state in LDS and the
// slot-scheduled sweep over a row.  Everything is in an anonymous namespace: each
// translation unit that includes it keeps its own copy.
#pragma once

#include <hip/hip_runtime.h>

#include <cfloat>
#include <cmath>
#include <cstdint>

#include "resispec.h"

namespace {


constexpr int kBlock = 512;              // threads per row workgroup (all-nodes schedule)
constexpr int kMaxWaves = 16;            // waves per workgroup at most
constexpr int kMaxCand = RS_MAX_CANDIDATES;
// 128-bit loads per lane and row in one chunk: bf16 rows (8 elements a load), fp32 rows
// (4 elements a load)
constexpr int kUnr16 = 2;
constexpr int kUnr32 = 2;
// Load policy.  Data whose last full use is the current pass is read with nontemporal
// loads (about 12% more streaming bandwidth on gfx950): pass 1 of rows without
// children and every rejection pass.  Pass 1 of a row with children uses ordinary loads,
// so a rejection pass that follows soon after can still find part of the row in the
// last-level cache.
constexpr bool kNtPass1 = false;
constexpr bool kNtRej = true;
constexpr bool kNtLeaf = true;
constexpr int kMaxSlots = 128;           // per-row slots (runs of chunks) with partial sums
// A row's exponent reference is fixed before pass 1; sums outside [2^-kLow, inf) send the
// row through an exact-maximum pass and a second pass 1.
constexpr double kLowSum = 1.0 / 1048576.0;

// ------------------------------------------------------------------ loads ----

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float widen(float x) { return x; }
__device__ __forceinline__ float widen(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// VEC consecutive elements starting at element idx, kept as raw words until used;
// elements at or beyond V read as -inf, which makes them contribute exactly zero to
// every sum below.
// 16-byte load; NT: nontemporal (streamed past the caches' normal allocation)
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
template <bool NT>
__device__ __forceinline__ uint4 ld16(const void* p) {
    if (NT) {
        const u32x4 r = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
        return make_uint4(r.x, r.y, r.z, r.w);
    }
    return *reinterpret_cast<const uint4*>(p);
}
template <bool NT>
__device__ __forceinline__ uint32_t ld4(const void* p) {
    if (NT) return __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p));
    return *reinterpret_cast<const uint32_t*>(p);
}
template <bool NT>
__device__ __forceinline__ uint32_t ld2(const void* p) {
    if (NT) return __builtin_nontemporal_load(reinterpret_cast<const uint16_t*>(p));
    return *reinterpret_cast<const uint16_t*>(p);
}

template <typename In, int VEC>
struct Vec;

template <>
struct Vec<float, 4> {
    using raw = uint4;
    template <bool NT = false>
    static __device__ __forceinline__ raw load(const float* __restrict__ row, int idx, int V) {
        if (idx < V) return ld16<NT>(row + idx);
        return make_uint4(0xff800000u, 0xff800000u, 0xff800000u, 0xff800000u);
    }
    template <bool NT = false>
    static __device__ __forceinline__ raw load_full(const float* __restrict__ row, int idx) {
        return ld16<NT>(row + idx);
    }
    static __device__ __forceinline__ void unpack(const raw& r, float (&v)[4]) {
        v[0] = __uint_as_float(r.x); v[1] = __uint_as_float(r.y);
        v[2] = __uint_as_float(r.z); v[3] = __uint_as_float(r.w);
    }
};

template <>
struct Vec<uint16_t, 8> {
    using raw = uint4;
    template <bool NT = false>
    static __device__ __forceinline__ raw load(const uint16_t* __restrict__ row, int idx, int V) {
        if (idx < V) return ld16<NT>(row + idx);
        return make_uint4(0xff80ff80u, 0xff80ff80u, 0xff80ff80u, 0xff80ff80u);
    }
    template <bool NT = false>
    static __device__ __forceinline__ raw load_full(const uint16_t* __restrict__ row, int idx) {
        return ld16<NT>(row + idx);
    }
    static __device__ __forceinline__ void unpack(const raw& r, float (&v)[8]) {
        v[0] = bf16_lo(r.x); v[1] = bf16_hi(r.x);
        v[2] = bf16_lo(r.y); v[3] = bf16_hi(r.y);
        v[4] = bf16_lo(r.z); v[5] = bf16_hi(r.z);
        v[6] = bf16_lo(r.w); v[7] = bf16_hi(r.w);
    }
};

template <>
struct Vec<float, 1> {
    using raw = uint32_t;
    template <bool NT = false>
    static __device__ __forceinline__ raw load(const float* __restrict__ row, int idx, int V) {
        return idx < V ? ld4<NT>(row + idx) : 0xff800000u;
    }
    template <bool NT = false>
    static __device__ __forceinline__ raw load_full(const float* __restrict__ row, int idx) {
        return ld4<NT>(row + idx);
    }
    static __device__ __forceinline__ void unpack(const raw& r, float (&v)[1]) { v[0] = __uint_as_float(r); }
};

template <>
struct Vec<uint16_t, 1> {
    using raw = uint32_t;
    template <bool NT = false>
    static __device__ __forceinline__ raw load(const uint16_t* __restrict__ row, int idx, int V) {
        return idx < V ? ld2<NT>(row + idx) << 16 : 0xff800000u;
    }
    template <bool NT = false>
    static __device__ __forceinline__ raw load_full(const uint16_t* __restrict__ row, int idx) {
        return ld2<NT>(row + idx) << 16;
    }
    static __device__ __forceinline__ void unpack(const raw& r, float (&v)[1]) { v[0] = __uint_as_float(r); }
};

// Unpacked elements of one vector (used outside the streaming passes).
template <typename In, int VEC>
__device__ __forceinline__ void load_vec(const In* __restrict__ row, int idx, int V, float (&v)[VEC]) {
    Vec<In, VEC>::unpack(Vec<In, VEC>::load(row, idx, V), v);
}

// v_exp_f32: 2^x; results below the normal range flush to zero (they are more than
// 2^-126 below the row maximum and carry no mass at fp32 resolution).
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// exponent l * c2 + K with c2 = c2h + c2l (both > 0; see base_params)
__device__ __forceinline__ float expo(float l, float c2h, float c2l, float K) {
    return fmaf(l, c2l, fmaf(l, c2h, K));
}

// ------------------------------------------------------------- wave ops ----

// Wave-wide reductions with DPP lane moves inside each 16-lane row (xor 1, xor 2,
// half-row mirror, row mirror), then the four row results combined in a fixed order
// from lanes 0, 16, 32, 48.  Every lane returns the same value.
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
    return __int_as_float(dpp_i<CTRL>(__float_as_int(v)));
}
template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
    const int lo = dpp_i<CTRL>(__double2loint(v));
    const int hi = dpp_i<CTRL>(__double2hiint(v));
    return __hiloint2double(hi, lo);
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

__device__ __forceinline__ float readlane_f(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ double readlane_d(double v, int l) {
    return __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(v), l),
                            __builtin_amdgcn_readlane(__double2loint(v), l));
}

__device__ __forceinline__ float wave_max(float v) {
    v = fmaxf(v, dpp_f<kDppXor1>(v));
    v = fmaxf(v, dpp_f<kDppXor2>(v));
    v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
    v = fmaxf(v, dpp_f<kDppMirror>(v));
    return fmaxf(fmaxf(readlane_f(v, 0), readlane_f(v, 16)), fmaxf(readlane_f(v, 32), readlane_f(v, 48)));
}

__device__ __forceinline__ double wave_sum(double v) {
    v += dpp_d<kDppXor1>(v);
    v += dpp_d<kDppXor2>(v);
    v += dpp_d<kDppHalfMirror>(v);
    v += dpp_d<kDppMirror>(v);
    return (readlane_d(v, 0) + readlane_d(v, 16)) + (readlane_d(v, 32) + readlane_d(v, 48));
}

// Inclusive prefix sum over the 64 lanes (fp64) with DPP moves: Hillis-Steele steps of
// 1, 2, 4 and 8 lanes inside each row of 16 lanes, then the last lane of rows 0 and 2
// added to rows 1 and 3 (row_bcast:15), then the last lane of row 1 added to rows 2 and 3
// (row_bcast:31).  The additions come in a fixed order, so every call gives the same
// bits.  Lanes with no source lane add zero.
template <int CTRL, int ROWMASK>
__device__ __forceinline__ double dpp_d_or_zero(double v) {
    const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), CTRL, ROWMASK, 0xF, true);
    const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), CTRL, ROWMASK, 0xF, true);
    return __hiloint2double(hi, lo);
}
constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118;
constexpr int kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143;

__device__ __forceinline__ double wave_incl_scan(double v, int) {
    v += dpp_d_or_zero<kDppRowShr1, 0xF>(v);
    v += dpp_d_or_zero<kDppRowShr2, 0xF>(v);
    v += dpp_d_or_zero<kDppRowShr4, 0xF>(v);
    v += dpp_d_or_zero<kDppRowShr8, 0xF>(v);
    v += dpp_d_or_zero<kDppRowBcast15, 0xA>(v);
    v += dpp_d_or_zero<kDppRowBcast31, 0xC>(v);
    return v;
}

// ------------------------------------------------------------ row state ----

struct Smem {
    int32_t status;
    int32_t decision;     // -1 continue, >= 0 accepted candidate, -2 fault
    int32_t next_slot;    // slot counter of the running sweep
    int32_t nt_hint;      // pass 1 may stream the rest of the row nontemporally (a cache hint)
    int32_t nc;           // rows with more nodes than threads only
    float ur;
    double St, Sd;        // sums of exp2(l c2 + K)
    int32_t wcount[kMaxWaves];
    int32_t wbad[kMaxWaves];
    int32_t cand_tok[kMaxCand];
    int32_t cand_node[kMaxCand];
    float cand_u[kMaxCand];
    float cand_lt[kMaxCand];
    float cand_ld[kMaxCand];
    double cand_p[kMaxCand];
    double cand_q[kMaxCand];
    // rejection steps, in test order; fp32 copies are in target-mass units
    int32_t st_x[kMaxCand + 1];
    float st_c[kMaxCand + 1];       // ResiSpec: Z * dscale * St/Sd.  Standard: C * St/Sd
    float st_a[kMaxCand + 1];       // ResiSpec: a
    float st_i[kMaxCand + 1];       // ResiSpec: 1/Z
    float st_k1[kMaxCand + 1];      // ResiSpec: a/Z
    float st_kc[kMaxCand + 1];      // ResiSpec: (1 - a) c/Z
    double st_zd[kMaxCand + 1], st_ad[kMaxCand + 1];
    double st_ds[kMaxCand + 1];     // draft scale (without replacement)
    double st_rx[kMaxCand + 1];     // R(x_i) of the tested candidate (normalised)
    // standard residual after i + 1 rejections, collapsed:
    //   R = max(p - C_i q, 0) / Tot_i,  C_i = C_{i-1} + Tot_{i-1} dscale_i
    double st_C[kMaxCand + 1], st_tot[kMaxCand + 1];
    // ResiSpec, first rejection: min(c Q, R) = 2^f0 exp2(min(aR - f0, aQ + e)) with
    // log2 c = e + f0; kq0 = Kd + e (integer valued)
    float st_f0, st_kq0;
    double st_2f0;                  // 2^f0 (as v_exp_f32 gives it)
    double rx0e;                    // the fp32 element value of R at x_0 (target units)
    int32_t sx0;                    // slot holding x_0
    double slotP[kMaxSlots];        // pass-1 slot totals of the target row
    uint32_t hit_slots[kMaxSlots / 32];  // slots that hold a rejected token
    // slots that hold a candidate (without replacement: pass 1 sums the draft row without
    // the candidates, whose masses are added in fp64, so the draft mass left after any
    // removals is a sum of what remains rather than a difference)
    uint32_t cand_slots[kMaxSlots / 32];
    double Sd_nc;                   // draft mass outside the candidates (without replacement)
    // per-lane partials of every slot of the running pass ([lane][slot], padded so a
    // wave's 64 stores hit 64 distinct banks), reduced after the pass in a fixed order
    float partA[64][kMaxSlots + 1];
    float partB[64][kMaxSlots + 1];
    double slotA[kMaxSlots];
    double slotB[kMaxSlots];
    double slotT[kMaxSlots];
    float wmax[2][kMaxWaves];
    // draw
    int32_t token;
    double total;
    int32_t group_ok;               // the last barrier of a row group completed in time
    // outcome of the row (path schedule)
    int32_t res_child, res_tok, res_status;
};

// Per-slot sums of the lane partials of a pass, in a fixed order, so the totals are
// bitwise reproducible whatever wave processed which slot, and whatever the block size.
// Stage 1 (the first NG * kMaxSlots threads, for the slots in [s_lo, s_hi)): thread t
// adds lanes [g*GS, g*GS + GS) of slot t % kMaxSlots, g = t / kMaxSlots, in fp64 and
// parks the sum in rows g*GS and g*GS + 1 of that column as two 32-bit halves (no other
// thread touches those cells).  Stage 2, after a barrier (slot_group_sum): the NG group
// sums of one slot are added in group order.
template <int BLK>
struct SlotGroups {
    static constexpr int NG = 4;
    static constexpr int GS = 64 / NG;
    static_assert(NG * kMaxSlots <= BLK, "the block must hold a thread per group and slot");
};

__device__ __forceinline__ void park_double(float (&part)[64][kMaxSlots + 1], int r, int s, double v) {
    const unsigned long long bits = (unsigned long long)__double_as_longlong(v);
    part[r][s] = __uint_as_float((uint32_t)bits);
    part[r + 1][s] = __uint_as_float((uint32_t)(bits >> 32));
}

template <int BLK>
__device__ __forceinline__ void slot_sums_stage1(Smem& sm, int s_lo, int s_hi, bool wantB) {
    using SG = SlotGroups<BLK>;
    const int s = threadIdx.x % kMaxSlots, g = threadIdx.x / kMaxSlots;
    if (g >= SG::NG || s < s_lo || s >= s_hi) return;
    double a = 0.0, c = 0.0;
#pragma unroll
    for (int l = 0; l < SG::GS; ++l) a += (double)sm.partA[g * SG::GS + l][s];
    if (wantB) {
#pragma unroll
        for (int l = 0; l < SG::GS; ++l) c += (double)sm.partB[g * SG::GS + l][s];
    }
    park_double(sm.partA, g * SG::GS, s, a);
    if (wantB) park_double(sm.partB, g * SG::GS, s, c);
}

// Stage 1 over one array of partials only (kernels with a single sum per slot).
template <int BLK>
__device__ __forceinline__ void slot_sums_stage1_one(float (&part)[64][kMaxSlots + 1], int s_lo, int s_hi) {
    using SG = SlotGroups<BLK>;
    const int s = threadIdx.x % kMaxSlots, g = threadIdx.x / kMaxSlots;
    if (g >= SG::NG || s < s_lo || s >= s_hi) return;
    double a = 0.0;
#pragma unroll
    for (int l = 0; l < SG::GS; ++l) a += (double)part[g * SG::GS + l][s];
    park_double(part, g * SG::GS, s, a);
}

template <int BLK>
__device__ __forceinline__ double slot_group_sum(const float (&part)[64][kMaxSlots + 1], int s) {
    using SG = SlotGroups<BLK>;
    double v = 0.0;
#pragma unroll
    for (int g = 0; g < SG::NG; ++g) {
        const uint32_t lo = __float_as_uint(part[g * SG::GS][s]);
        const uint32_t hi = __float_as_uint(part[g * SG::GS + 1][s]);
        v += __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
    }
    return v;
}

// Exponent reference for a maximum m: an integer-valued float near -m * c2, so that
// the fp32 exponents near the maximum are small and exactly offset, and a shift of
// the reference by an integer (the first-rejection split of log2 c) stays exact.
__device__ __forceinline__ float kref(float m, float c2h) {
    return m > -FLT_MAX ? -ceilf(m * c2h) : 0.0f;
}

// One chunk (UNR loads of 64 * VEC elements per row) starting at element c0 + lane * VEC;
// chunks wholly below V load without per-lane bounds checks.
template <typename In, int VEC, int UNR, bool PAIR, bool NT>
__device__ __forceinline__ void load_chunk(const In* __restrict__ tg, const In* __restrict__ dg,
                                           int c0, int V, typename Vec<In, VEC>::raw (&t)[UNR],
                                           typename Vec<In, VEC>::raw (&d)[UNR]) {
    using W = Vec<In, VEC>;
    constexpr int CHUNK = 64 * VEC * UNR;
    const int l0 = c0 + (threadIdx.x & 63) * VEC;
    if (c0 + CHUNK <= V) {
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            t[u] = W::template load_full<NT>(tg, l0 + u * 64 * VEC);
            if (PAIR) d[u] = W::template load_full<NT>(dg, l0 + u * 64 * VEC);
        }
    } else {
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            t[u] = W::template load<NT>(tg, l0 + u * 64 * VEC, V);
            if (PAIR) d[u] = W::template load<NT>(dg, l0 + u * 64 * VEC, V);
        }
    }
}

// One pass over the row.  The row is cut into chunks of 64 * VEC * UNR elements (one
// 128-bit load per lane and UNR) and runs of G chunks form slots.  Waves take slots
// from a shared counter, so the eight waves of the block finish within about one chunk
// of each other; a wave's first slot is its own index, so its first loads can be
// issued before the counter is set (PRE = 1: its target part was loaded by the caller
// into pre_t; PRE = 2: target and draft parts, into pre_t and pre_d).  Two register
// sets alternate: the next chunk is loaded into one while the other is processed (four
// for one row with RING4, below).
// body(t, d, idx0, slot) gets the unpacked elements
// of a chunk (element (u, e) has index idx0 + u * 64 * VEC + e); flush(slot) runs
// after a slot's last chunk.  reverse: slots in descending order, chunks descending
// inside a slot.  The sweep covers slots [sbase, sbase + nslots) of the row (a share of
// them when several workgroups verify one row; the waves' first slots are sbase + w).
//
// nt_hint (ordinary loads only, NT = false): a shared flag that a wave reads each time it
// takes a slot; once it is set, the wave's further loads are nontemporal.  Only the cache
// policy changes, never the elements or their order.
template <typename In, int VEC, int UNR, bool PAIR, int PRE, bool NT, bool RING4 = false, typename Body,
          typename Flush>
__device__ __forceinline__ void wave_sweep(const In* __restrict__ tg, const In* __restrict__ dg,
                                           int V, int G, int nslots, int sbase, bool reverse,
                                           const typename Vec<In, VEC>::raw (&pre_t)[UNR],
                                           const typename Vec<In, VEC>::raw (&pre_d)[UNR],
                                           int* counter, Body&& body, Flush&& flush,
                                           const int32_t* nt_hint = nullptr) {
    using W = Vec<In, VEC>;
    using raw = typename W::raw;
    constexpr int CHUNK = 64 * VEC * UNR;
    const int lane = threadIdx.x & 63;
    const int wid = threadIdx.x >> 6;
    const int lane0 = lane * VEC;
    // first element of chunk j of a slot (the same for every lane)
    auto chunk_start = [&](int slot, int j) -> int {
        return (slot * G + (reverse ? G - 1 - j : j)) * CHUNK;
    };
    int slot = wid < nslots ? sbase + (reverse ? nslots - 1 - wid : wid) : -1;
    if (slot < 0) return;
    // the counter is read one slot ahead, so its latency overlaps a chunk's work
    bool nt_now = false;
    auto take = [&]() -> int {
        int v = 0;
        if (lane == 0) v = atomicAdd(counter, 1);
        v = __builtin_amdgcn_readfirstlane(v);
        if (!NT && nt_hint) nt_now = __builtin_amdgcn_readfirstlane(*nt_hint) != 0;
        return v < nslots ? sbase + (reverse ? nslots - 1 - v : v) : -1;
    };
    int ahead = take();
    auto advance = [&](int& s, int& j) {
        if (++j == G) {
            s = ahead;
            j = 0;
            if (s >= 0) ahead = take();
        }
    };
    auto load = [&](int s, int j, raw (&t)[UNR], raw (&d)[UNR]) {
        if (!NT && nt_now)
            load_chunk<In, VEC, UNR, PAIR, true>(tg, dg, chunk_start(s, j), V, t, d);
        else
            load_chunk<In, VEC, UNR, PAIR, NT>(tg, dg, chunk_start(s, j), V, t, d);
    };
    auto process = [&](const raw (&ct)[UNR], const raw (&cd)[UNR], int s, int j) {
        float t[UNR][VEC], d[UNR][VEC];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            W::unpack(ct[u], t[u]);
            if (PAIR) W::unpack(cd[u], d[u]);
        }
        body(t, d, chunk_start(s, j) + lane0, s);
        if (j == G - 1) flush(s);
    };
    if constexpr (!PAIR && RING4) {
        // One row, RING4: the registers of the draft half hold two more chunks, so three
        // chunks are in flight while one is processed.  A buffer is refilled, with the
        // chunk after the last one requested, as soon as it has been processed; chunks
        // are processed in the same order as with two buffers.  (Measured: 1% faster
        // verification of the mostly-leaf serving batch, 3% slower in the draft step,
        // whose waves also draw.)
        raw b0[UNR], b1[UNR], b2[UNR], b3[UNR];
        int p0 = slot, k0 = 0, p1, k1, p2, k2, p3, k3;
        if (PRE >= 1) {
#pragma unroll
            for (int u = 0; u < UNR; ++u) b0[u] = pre_t[u];
        } else {
            load(p0, k0, b0, b0);
        }
        int ls = p0, lj = 0;   // the last chunk requested (slot -1: none left)
        auto refill = [&](raw (&b)[UNR], int& ps, int& pj) {
            if (ls >= 0) advance(ls, lj);
            ps = ls;
            pj = lj;
            if (ps >= 0) load(ps, pj, b, b);
        };
        refill(b1, p1, k1);
        refill(b2, p2, k2);
        refill(b3, p3, k3);
        for (;;) {
            process(b0, b0, p0, k0);
            refill(b0, p0, k0);
            if (p1 < 0) break;
            process(b1, b1, p1, k1);
            refill(b1, p1, k1);
            if (p2 < 0) break;
            process(b2, b2, p2, k2);
            refill(b2, p2, k2);
            if (p3 < 0) break;
            process(b3, b3, p3, k3);
            refill(b3, p3, k3);
            if (p0 < 0) break;
        }
        return;
    }
    raw at[UNR], ad[UNR], bt[UNR], bd[UNR];
    int sa = slot, ja = 0;
    if (PRE >= 1) {
#pragma unroll
        for (int u = 0; u < UNR; ++u) at[u] = pre_t[u];
        if (PAIR) {
            if (PRE == 2) {
#pragma unroll
                for (int u = 0; u < UNR; ++u) ad[u] = pre_d[u];
            } else {
                const int c0 = chunk_start(sa, 0);
#pragma unroll
                for (int u = 0; u < UNR; ++u) ad[u] = W::template load<NT>(dg, c0 + lane0 + u * 64 * VEC, V);
            }
        }
    } else {
        load(sa, ja, at, ad);
    }
    for (;;) {
        int sb = sa, jb = ja;
        advance(sb, jb);
        if (sb >= 0) load(sb, jb, bt, bd);
        process(at, ad, sa, ja);
        if (sb < 0) break;
        sa = sb;
        ja = jb;
        advance(sa, ja);
        if (sa >= 0) load(sa, ja, at, ad);
        process(bt, bd, sb, jb);
        if (sa < 0) break;
    }
}

// ------------------------------------------------------------------- host ----

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline rs_status check_params(const rs_params* prm) {
    if (!prm) return RS_ERR_INVALID_ARG;
    if (prm->mode != RS_MODE_RESISPEC && prm->mode != RS_MODE_SPECINFER) return RS_ERR_INVALID_ARG;
    if (prm->logits_dtype != RS_F32 && prm->logits_dtype != RS_BF16) return RS_ERR_INVALID_ARG;
    if (!(prm->temperature > 0.0f) || !std::isfinite(prm->temperature)) return RS_ERR_INVALID_ARG;
    return RS_OK;
}

// log2(e) / T as c2h + c2l with c2h strictly below it, so c2l > 0: a -inf logit then
// gives the exponent -inf (never -inf + inf) and contributes exactly zero.
inline void split_c2(float temperature, float* c2h_out, float* c2l_out) {
    const double c2 = 1.4426950408889634 / (double)temperature;
    float c2h = (float)c2;
    if ((double)c2h >= c2) c2h = std::nextafter(c2h, 0.0f);
    *c2h_out = c2h;
    *c2l_out = (float)(c2 - (double)c2h);
}

}  // namespace
