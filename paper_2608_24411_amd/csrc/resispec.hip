// resispec.hip -- gfx950 kernels and C ABI of the ResiSpec verification step.
//
// Paper: "ResiSpec: Enhancing Multi-Candidate Speculative Sampling via Residual
// Distribution Shaping".  One workgroup verifies one tree node (one logits row):
//
//   pass 1   online softmax statistics (max, sum of exp) of the target row and, for
//            nodes with children, the draft row (Preliminary; temperature T);
//   tests    candidate i is accepted iff u_i < R_i(x_i) / D_i(x_i) (Eq. 2 and
//            Algorithm 1), evaluated in fp64 on the gathered candidate logits;
//   pass i+1 after the i-th rejection one more pass over the row computes the sums the
//            residual update needs:
//              standard (Eq. 1/2):   S = sum_j max(R_j - D_j, 0)
//              ResiSpec (Algorithm 1, GetProxy): M = sum_{j != x0} min(Z D_j, R_j) and
//                                    SR = sum_{j != x0} R_j, with Z = D(x0) - R(x0).
//            GetProxy's one-shot redistribution of Delta = Z - M into the capacity
//            R_j - m_j gives, with a = Delta / (SR - M), the residual
//              R'_j = ((1 - a) min(Z D_j, R_j) + a R_j) / Z   (j != x0),   R'_x0 = 0,
//            i.e. norm(max(R - K, 0)) for the proxy K = R - r, K(x0) = D(x0).  So the
//            residual is never materialised: every pass re-derives R_j from the two
//            logits of token j through the chain of per-rejection scalars;
//   draw     when every candidate is rejected (or the node is a leaf: bonus draw from
//            p), the token is the smallest j whose running sum of the final residual in
//            vocabulary order exceeds u * total.  The last pass records per-tile partial
//            sums, so the draw re-reads a single tile.
//
// Numerics: elements in fp32 (bf16 widened exactly), every sum accumulated in fp64,
// the candidates' probabilities and the scalar chain in fp64.  Exponents are taken as
// exp2(l * c2 + K) with c2 = log2(e)/T split into two floats and K = -max * c2 rounded
// once; the rounding of K is common to a whole row and cancels in the normalisation,
// and the fp64 gathers use the same constants, so candidate probabilities agree with
// the fp32 sums they are divided by.  Residual elements are carried in units of the
// target row's unnormalised mass (the target normaliser is folded into the step
// constants).
//
// A second kernel walks each tree from the root along accepted children.

#include <hip/hip_runtime.h>

#include <cfloat>
#include <cmath>
#include <cstdint>

#include "resispec.h"

namespace {

constexpr int kBlock = 512;
constexpr int kWaves = kBlock / 64;
constexpr int kMaxCand = RS_MAX_CANDIDATES;
constexpr int kMaxTiles = 64;

// ------------------------------------------------------------------ loads ----

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float widen(float x) { return x; }
__device__ __forceinline__ float widen(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// VEC consecutive elements starting at element idx, kept as raw words until used;
// elements at or beyond V read as -inf, which makes them contribute exactly zero to
// every sum below.
template <typename In, int VEC>
struct Vec;

template <>
struct Vec<float, 4> {
    using raw = uint4;
    static __device__ __forceinline__ raw load(const float* __restrict__ row, int idx, int V) {
        if (idx < V) return *reinterpret_cast<const uint4*>(row + idx);
        return make_uint4(0xff800000u, 0xff800000u, 0xff800000u, 0xff800000u);
    }
    static __device__ __forceinline__ void unpack(const raw& r, float (&v)[4]) {
        v[0] = __uint_as_float(r.x); v[1] = __uint_as_float(r.y);
        v[2] = __uint_as_float(r.z); v[3] = __uint_as_float(r.w);
    }
};

template <>
struct Vec<uint16_t, 8> {
    using raw = uint4;
    static __device__ __forceinline__ raw load(const uint16_t* __restrict__ row, int idx, int V) {
        if (idx < V) return *reinterpret_cast<const uint4*>(row + idx);
        return make_uint4(0xff80ff80u, 0xff80ff80u, 0xff80ff80u, 0xff80ff80u);
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
    static __device__ __forceinline__ raw load(const float* __restrict__ row, int idx, int V) {
        return idx < V ? __float_as_uint(row[idx]) : 0xff800000u;
    }
    static __device__ __forceinline__ void unpack(const raw& r, float (&v)[1]) { v[0] = __uint_as_float(r); }
};

template <>
struct Vec<uint16_t, 1> {
    using raw = uint32_t;
    static __device__ __forceinline__ raw load(const uint16_t* __restrict__ row, int idx, int V) {
        return idx < V ? ((uint32_t)row[idx]) << 16 : 0xff800000u;
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

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ double wave_incl_scan(double v, int lane) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const double n = __shfl_up(v, o, 64);
        if (lane >= o) v += n;
    }
    return v;
}

// ------------------------------------------------------------ row state ----

struct Smem {
    int32_t status;
    int32_t nc;
    int32_t decision;     // -1 continue, >= 0 accepted candidate, -2 fault
    float ur;
    float Kt, Kd;         // exponent offsets -max * c2 of target / draft
    double St, Sd;        // sums of exp2(l c2 + K)
    int32_t cand_tok[kMaxCand];
    int32_t cand_node[kMaxCand];
    float cand_u[kMaxCand];
    float cand_lt[kMaxCand];
    float cand_ld[kMaxCand];
    double cand_p[kMaxCand];
    double cand_q[kMaxCand];
    // rejection steps, in test order; fp32 copies are in target-mass units
    int32_t st_x[kMaxCand + 1];
    int32_t st_iter[kMaxCand + 1];  // loop iteration that holds token x
    float st_c[kMaxCand + 1];       // ResiSpec: Z * dscale * St/Sd.  Standard: dscale * St/Sd
    float st_a[kMaxCand + 1];       // ResiSpec: a
    float st_i[kMaxCand + 1];       // ResiSpec: 1/Z.  Standard: 1/S
    double st_zd[kMaxCand + 1], st_ad[kMaxCand + 1], st_id[kMaxCand + 1];
    double st_ds[kMaxCand + 1];     // draft scale (without replacement)
    // per-tile partials written by one wave each
    double tpA[kMaxTiles][kWaves];
    double tpB[kMaxTiles][kWaves];
    float tpK[kMaxTiles][kWaves];
    double tileT[kMaxTiles];
    // cross-wave reductions
    float redm[2][kWaves];
    float redk[2][kWaves];
    double reds[2][kWaves];
    double scan_w[kWaves];
    int32_t first_w[kWaves + 1];
    // draw
    int32_t ksel;
    double base, thr, total;
    int32_t token;
};

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
    int32_t B, N;
    int32_t V;
    float T;
    float c2h, c2l;      // log2(e) / T = c2h + c2l
    int32_t worep, bonus, flat;
    int32_t niters;      // loop iterations per pass
    int32_t tile_iters;  // loop iterations per tile
    int32_t ntiles;
};

__device__ __forceinline__ float kref(float m, float c2h) {
    return m > -FLT_MAX ? -(m * c2h) : 0.0f;
}

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
    for (int j = threadIdx.x; j < P.V; j += kBlock) out[j] = 0.0f;
}

// Rejection-step terms of one element, given its target mass R (target units) and
// unnormalised draft mass Q.  The chain over the earlier steps 0..i-1 first.
//   standard: A = max(R - c_i Q, 0)                    (c_i = dscale_i St/Sd)
//   ResiSpec: A = min(c_i Q, R), B = R, both 0 at x_i   (c_i = Z_i dscale_i St/Sd)
// CHECK = false skips the token comparisons (no rejected token in this element's
// loop iteration); the standard update needs none: R < D at every rejected token.
template <int MODE, bool CHECK>
__device__ __forceinline__ void chain_terms(float R, float Q, int j, const Smem& sm, int i,
                                            float& A, float& Bv) {
    for (int t = 0; t < i; ++t) {
        const float c = sm.st_c[t];
        if (MODE == RS_MODE_SPECINFER) {
            R = fmaxf(fmaf(-c, Q, R), 0.0f) * sm.st_i[t];
        } else {
            const float m = fminf(c * Q, R);
            R = fmaf(sm.st_a[t], R - m, m) * sm.st_i[t];
            if (CHECK && j == sm.st_x[t]) R = 0.0f;
        }
    }
    const float c = sm.st_c[i];
    if (MODE == RS_MODE_SPECINFER) {
        A = fmaxf(fmaf(-c, Q, R), 0.0f);
        Bv = 0.0f;
    } else {
        const bool x0 = CHECK && j == sm.st_x[i];
        A = x0 ? 0.0f : fminf(c * Q, R);
        Bv = x0 ? 0.0f : R;
    }
}

// Scalar chain for the accept test of candidate i (fp64, normalised units).
template <int MODE>
__device__ double scalar_residual(const Smem& sm, int i, double p, double q, int32_t x,
                                  bool worep, double& Dout) {
    double R = p;
    bool removed = false;
    for (int t = 0; t < i; ++t) {
        const double Dt = removed ? 0.0 : q * sm.st_ds[t];
        if (MODE == RS_MODE_SPECINFER) {
            const double w = R - Dt;
            R = (w > 0.0 ? w : 0.0) * sm.st_id[t];
        } else {
            if (x == sm.st_x[t]) {
                R = 0.0;
            } else {
                const double zd = sm.st_zd[t] * Dt;
                const double m = zd < R ? zd : R;
                R = ((1.0 - sm.st_ad[t]) * m + sm.st_ad[t] * R) / sm.st_zd[t];
            }
        }
        if (worep && x == sm.st_x[t]) removed = true;
    }
    Dout = removed ? 0.0 : q * sm.st_ds[i];
    return R;
}

// One sweep over the row with register prefetch of the next iteration.  body(t, d,
// idx0, it) gets the UNR x VEC unpacked elements of iteration `it`; element (u, e)
// has index idx0 + u * kBlock * VEC + e.  flush(tile) runs after the last iteration
// of a tile.
template <typename In, int VEC, int UNR, bool PAIR, typename Body, typename Flush>
__device__ __forceinline__ void sweep(const In* __restrict__ tg, const In* __restrict__ dg,
                                      int V, int niters, int ti, bool reverse, Body&& body,
                                      Flush&& flush) {
    using W = Vec<In, VEC>;
    using raw = typename W::raw;
    constexpr int ITER = kBlock * VEC * UNR;
    const int lane0 = threadIdx.x * VEC;
    raw ct[UNR], cd[UNR];
    int it = reverse ? niters - 1 : 0;
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
        ct[u] = W::load(tg, it * ITER + u * kBlock * VEC + lane0, V);
        if (PAIR) cd[u] = W::load(dg, it * ITER + u * kBlock * VEC + lane0, V);
    }
    int tile = it / ti;
    int edge = reverse ? tile * ti : min((tile + 1) * ti, niters) - 1;
    for (int k = 0; k < niters; ++k) {
        const int nit = reverse ? it - 1 : it + 1;
        raw nt[UNR], nd[UNR];
        if (k + 1 < niters) {
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                nt[u] = W::load(tg, nit * ITER + u * kBlock * VEC + lane0, V);
                if (PAIR) nd[u] = W::load(dg, nit * ITER + u * kBlock * VEC + lane0, V);
            }
        }
        float t[UNR][VEC], d[UNR][VEC];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            W::unpack(ct[u], t[u]);
            if (PAIR) W::unpack(cd[u], d[u]);
        }
        body(t, d, it * ITER + lane0, it);
        if (it == edge) {
            flush(tile);
            tile += reverse ? -1 : 1;
            edge = reverse ? tile * ti : min((tile + 1) * ti, niters) - 1;
        }
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            ct[u] = nt[u];
            if (PAIR) cd[u] = nd[u];
        }
        it = nit;
    }
}

// ------------------------------------------------------------ row kernel ----

template <typename In, int VEC, int UNR, int MODE>
__global__ void __launch_bounds__(kBlock) rs_row_kernel(const KParams P) {
    __shared__ Smem sm;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int V = P.V;
    constexpr int ITER = kBlock * VEC * UNR;

    int64_t row;
    int32_t b, n;
    if (P.flat) {
        row = blockIdx.x;
        b = (int32_t)row;
        n = 0;
    } else {
        // node-major order: the roots of all sequences first, then node 1, ... (nodes
        // with children come early in a topological numbering)
        const int32_t g = blockIdx.x;
        n = g / P.B;
        b = g - n * P.B;
        row = (int64_t)b * P.N + n;
    }
    const In* __restrict__ tg = reinterpret_cast<const In*>(P.tgt) + row * V;
    const In* __restrict__ dg = reinterpret_cast<const In*>(P.dft) + row * V;

    // ---- row description: candidates, their uniforms and logits, structural checks
    if (tid == 0) {
        sm.status = RS_SEQ_OK;
        sm.nc = 0;
        sm.decision = -1;
    }
    __syncthreads();
    if (P.flat) {
        if (tid < P.k) {
            const int32_t x = P.cand_ids[row * P.k + tid];
            sm.cand_tok[tid] = x;
            sm.cand_u[tid] = P.ua_flat[row * P.k + tid];
            sm.cand_node[tid] = tid;
            const bool ok = x >= 0 && x < V;
            sm.cand_lt[tid] = ok ? widen(tg[x]) : 0.0f;
            sm.cand_ld[tid] = ok ? widen(dg[x]) : 0.0f;
        }
        if (tid == 0) {
            sm.nc = P.k;
            sm.ur = P.ur_flat[row];
        }
        __syncthreads();
    } else {
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
                    }
                }
                count += __popcll(mask);
            }
            if (lane == 0) {
                sm.nc = count;
                sm.ur = P.ur[row];
                if (bad) sm.status = RS_SEQ_BAD_TREE;
                else if (count > kMaxCand) sm.status = RS_SEQ_TOO_MANY_CHILDREN;
            }
        }
        __syncthreads();
    }
    const int nc = sm.nc;
    if (sm.status != RS_SEQ_OK) {
        if (tid == 0) write_outcome(P, row, -1, -1, sm.status);
        zero_residual_row(P, row);
        return;
    }
    if (nc == 0 && !P.flat && !P.bonus) {
        if (tid == 0) write_outcome(P, row, -1, -1, RS_SEQ_OK);
        zero_residual_row(P, row);
        return;
    }

    const bool internal = nc > 0;
    const float c2h = P.c2h, c2l = P.c2l;
    const int niters = P.niters, ti = P.tile_iters;

    // ---- pass 1: softmax statistics (per-lane running max; sums rescaled exactly
    // when the reference K = -max * c2 moves)
    {
        float mt = -FLT_MAX, kt = 0.0f, md = -FLT_MAX, kd = 0.0f;
        double st = 0.0, sd = 0.0;
        float stile = 0.0f;   // leaf rows: this tile's share of st (reference kt)
        auto flush = [&](int tile) {
            if (internal) return;
            const float mw = wave_max(mt);
            const float kw = kref(mw, c2h);
            const double sw = wave_sum(stile > 0.0f ? (double)stile * exp2((double)kw - (double)kt) : 0.0);
            if (lane == 0) {
                sm.tpK[tile][wid] = kw;
                sm.tpA[tile][wid] = sw;
            }
            stile = 0.0f;
        };
        if (internal) {
            sweep<In, VEC, UNR, true>(tg, dg, V, niters, ti, false,
                [&](const float (&t)[UNR][VEC], const float (&d)[UNR][VEC], int, int) {
                    float mx = -FLT_MAX, my = -FLT_MAX;
#pragma unroll
                    for (int u = 0; u < UNR; ++u)
#pragma unroll
                        for (int e = 0; e < VEC; ++e) {
                            mx = fmaxf(mx, t[u][e]);
                            my = fmaxf(my, d[u][e]);
                        }
                    if (mx > mt) {
                        const float nk = -(mx * c2h);
                        st *= exp2((double)nk - (double)kt);
                        mt = mx;
                        kt = nk;
                    }
                    if (my > md) {
                        const float nk = -(my * c2h);
                        sd *= exp2((double)nk - (double)kd);
                        md = my;
                        kd = nk;
                    }
                    float a = 0.0f, c = 0.0f;
#pragma unroll
                    for (int u = 0; u < UNR; ++u)
#pragma unroll
                        for (int e = 0; e < VEC; ++e) {
                            a += exp2_fast(expo(t[u][e], c2h, c2l, kt));
                            c += exp2_fast(expo(d[u][e], c2h, c2l, kd));
                        }
                    st += (double)a;
                    sd += (double)c;
                },
                flush);
        } else {
            sweep<In, VEC, UNR, false>(tg, dg, V, niters, ti, false,
                [&](const float (&t)[UNR][VEC], const float (&)[UNR][VEC], int, int) {
                    float mx = -FLT_MAX;
#pragma unroll
                    for (int u = 0; u < UNR; ++u)
#pragma unroll
                        for (int e = 0; e < VEC; ++e) mx = fmaxf(mx, t[u][e]);
                    if (mx > mt) {
                        const float nk = -(mx * c2h);
                        const double f = exp2((double)nk - (double)kt);
                        st *= f;
                        stile = (float)(stile * f);
                        mt = mx;
                        kt = nk;
                    }
                    float a = 0.0f;
#pragma unroll
                    for (int u = 0; u < UNR; ++u)
#pragma unroll
                        for (int e = 0; e < VEC; ++e) a += exp2_fast(expo(t[u][e], c2h, c2l, kt));
                    st += (double)a;
                    stile += a;
                },
                flush);
        }
        // combine lanes, then waves (wave 0)
        {
            const float mw = wave_max(mt);
            const float kw = kref(mw, c2h);
            const double sw = wave_sum(st > 0.0 ? st * exp2((double)kw - (double)kt) : 0.0);
            float mw2 = -FLT_MAX, kw2 = 0.0f;
            double sw2 = 0.0;
            if (internal) {
                mw2 = wave_max(md);
                kw2 = kref(mw2, c2h);
                sw2 = wave_sum(sd > 0.0 ? sd * exp2((double)kw2 - (double)kd) : 0.0);
            }
            if (lane == 0) {
                sm.redm[0][wid] = mw;
                sm.redk[0][wid] = kw;
                sm.reds[0][wid] = sw;
                sm.redm[1][wid] = mw2;
                sm.redk[1][wid] = kw2;
                sm.reds[1][wid] = sw2;
            }
        }
        __syncthreads();
        if (wid == 0) {
            const bool in = lane < kWaves;
            const int w = in ? lane : 0;
            const float m0 = wave_max(in ? sm.redm[0][w] : -FLT_MAX);
            const float m1 = wave_max(in ? sm.redm[1][w] : -FLT_MAX);
            const float k0 = kref(m0, c2h), k1 = kref(m1, c2h);
            const double s0 = wave_sum(in && sm.reds[0][w] > 0.0
                                           ? sm.reds[0][w] * exp2((double)k0 - (double)sm.redk[0][w]) : 0.0);
            const double s1 = wave_sum(in && sm.reds[1][w] > 0.0
                                           ? sm.reds[1][w] * exp2((double)k1 - (double)sm.redk[1][w]) : 0.0);
            if (lane == 0) {
                sm.Kt = k0;
                sm.Kd = k1;
                sm.St = s0;
                sm.Sd = s1;
                if (!(s0 > 0.0) || (internal && !(s1 > 0.0))) sm.status = RS_SEQ_UNDERFLOW;
                sm.st_ds[0] = 1.0;
            }
        }
        __syncthreads();
        if (sm.status != RS_SEQ_OK) {
            if (tid == 0) write_outcome(P, row, -1, -1, sm.status);
            zero_residual_row(P, row);
            return;
        }
    }

    const double c2d = (double)c2h + (double)c2l;
    const float Kt = sm.Kt, Kd = sm.Kd;
    const double St = sm.St, Sd = sm.Sd;
    // draft mass in target units: q St / Sd, folded into the step constants
    const double q2t = internal ? St / Sd : 0.0;

    // ---- candidate probabilities in fp64, with the same exponent constants
    if (tid < nc) {
        const int32_t x = sm.cand_tok[tid];
        double pc = 0.0, qc = 0.0;
        if (x >= 0 && x < V) {
            pc = exp2((double)sm.cand_lt[tid] * c2d + (double)Kt) / St;
            qc = exp2((double)sm.cand_ld[tid] * c2d + (double)Kd) / Sd;
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
                double Dx;
                const double Rx = scalar_residual<MODE>(sm, i, sm.cand_p[i], sm.cand_q[i], x, worep, Dx);
                if (!(Dx > 0.0)) {
                    sm.status = RS_SEQ_ZERO_DRAFT;
                    dec = -2;
                } else if ((double)u < Rx / Dx) {
                    dec = i;
                } else {
                    const double z = Dx - Rx;   // ResiSpec budget
                    sm.st_x[i] = x;
                    sm.st_iter[i] = x / ITER;
                    sm.st_zd[i] = z;
                    sm.st_c[i] = (float)((MODE == RS_MODE_SPECINFER ? 1.0 : z) * sm.st_ds[i] * q2t);
                }
            }
            sm.decision = dec;
        }
        __syncthreads();
        if (sm.decision != -1) break;

        // rejection pass: sums of step i with per-tile partials
        {
            double accA = 0.0, accB = 0.0;   // this tile's lane partials
            auto flush = [&](int tile) {
                const double wa = wave_sum(accA);
                const double wb = (MODE == RS_MODE_RESISPEC) ? wave_sum(accB) : 0.0;
                if (lane == 0) {
                    sm.tpA[tile][wid] = wa;
                    sm.tpB[tile][wid] = wb;
                }
                accA = accB = 0.0;
            };
            const bool reverse = (i & 1) == 0;   // re-read the most recently fetched end first
            const int ii = i;
            sweep<In, VEC, UNR, true>(tg, dg, V, niters, ti, reverse,
                [&](const float (&t)[UNR][VEC], const float (&d)[UNR][VEC], int idx0, int it) {
                    bool hit = false;
                    if (MODE == RS_MODE_RESISPEC) {
                        for (int s = 0; s <= ii; ++s) hit |= (sm.st_iter[s] == it);
                    }
                    float fa = 0.0f, fb = 0.0f;
                    if (!hit) {
#pragma unroll
                        for (int u = 0; u < UNR; ++u)
#pragma unroll
                            for (int e = 0; e < VEC; ++e) {
                                const float R = exp2_fast(expo(t[u][e], c2h, c2l, Kt));
                                const float Q = exp2_fast(expo(d[u][e], c2h, c2l, Kd));
                                float A, Bv;
                                chain_terms<MODE, false>(R, Q, 0, sm, ii, A, Bv);
                                fa += A;
                                fb += Bv;
                            }
                    } else {
#pragma unroll
                        for (int u = 0; u < UNR; ++u)
#pragma unroll
                            for (int e = 0; e < VEC; ++e) {
                                const float R = exp2_fast(expo(t[u][e], c2h, c2l, Kt));
                                const float Q = exp2_fast(expo(d[u][e], c2h, c2l, Kd));
                                float A, Bv;
                                chain_terms<MODE, true>(R, Q, idx0 + u * kBlock * VEC + e, sm, ii, A, Bv);
                                fa += A;
                                fb += Bv;
                            }
                    }
                    accA += (double)fa;
                    accB += (double)fb;
                },
                flush);
        }
        __syncthreads();
        if (wid == 0) {
            double A = 0.0, Bv = 0.0;
            if (lane < P.ntiles) {
                for (int w = 0; w < kWaves; ++w) {
                    A += sm.tpA[lane][w];
                    Bv += sm.tpB[lane][w];
                }
            }
            // lane 0's sums, so that every lane derives identical constants
            const double totA = __shfl(wave_sum(A), 0, 64) / St;   // normalised units
            const double totB = __shfl(wave_sum(Bv), 0, 64) / St;
            const double z = sm.st_zd[i];
            double a = 0.0, inv;
            if (MODE == RS_MODE_SPECINFER) {
                inv = 1.0 / totA;
            } else {
                const double delta = z - totA;   // GetProxy deficit
                const double C = totB - totA;    // remaining capacity, x0 excluded
                a = (C > 0.0) ? delta / C : 0.0;
                inv = 1.0 / z;
            }
            if (lane < P.ntiles) {
                // tile totals of the unnormalised next residual (linear in the partials)
                sm.tileT[lane] = (MODE == RS_MODE_SPECINFER) ? A : (1.0 - a) * A + a * Bv;
            }
            if (lane == 0) {
                if (MODE == RS_MODE_SPECINFER && !(totA > 0.0)) {
                    sm.status = RS_SEQ_UNDERFLOW;
                    sm.decision = -2;
                }
                sm.st_ad[i] = a;
                sm.st_a[i] = (float)a;
                sm.st_id[i] = inv;
                sm.st_i[i] = (float)inv;
                if (worep) {
                    const double rest = 1.0 - sm.cand_q[i] * sm.st_ds[i];
                    sm.st_ds[i + 1] = rest > 0.0 ? sm.st_ds[i] / rest : 0.0;
                } else {
                    sm.st_ds[i + 1] = 1.0;
                }
            }
        }
        __syncthreads();
        if (sm.decision == -2) break;
    }

    if (sm.decision == -2) {
        if (tid == 0) write_outcome(P, row, -1, -1, sm.status);
        zero_residual_row(P, row);
        return;
    }
    if (sm.decision >= 0) {
        if (tid == 0) {
            const int d = sm.decision;
            write_outcome(P, row, sm.cand_node[d], sm.cand_tok[d], RS_SEQ_OK);
        }
        zero_residual_row(P, row);
        return;
    }

    // ---- every candidate rejected, or no candidates: inverse-CDF draw
    const float u = sm.ur;
    if (!(u >= 0.0f && u < 1.0f)) {
        if (tid == 0) write_outcome(P, row, -1, -1, RS_SEQ_BAD_UNIFORM);
        zero_residual_row(P, row);
        return;
    }
    const int last = nc - 1;   // index of the last rejection step (internal rows)
    if (wid == 0) {
        double T = 0.0;
        if (lane < P.ntiles) {
            if (internal) {
                T = sm.tileT[lane];
            } else {
                for (int w = 0; w < kWaves; ++w) {
                    const double s = sm.tpA[lane][w];
                    if (s > 0.0) T += s * exp2((double)Kt - (double)sm.tpK[lane][w]);
                }
            }
        }
        const double cum = wave_incl_scan(T, lane);
        const double total = __shfl(cum, 63, 64);
        const double thr = (double)u * total;
        const uint64_t hit = __ballot(lane < P.ntiles && cum > thr);
        int k = hit ? (__ffsll((unsigned long long)hit) - 1) : -1;
        if (k < 0) {   // rounding guard: last tile with mass
            const uint64_t pos = __ballot(lane < P.ntiles && T > 0.0);
            k = pos ? 63 - __clzll((long long)pos) : 0;
        }
        const double excl = cum - T;
        const double base = __shfl(excl, k, 64);
        if (lane == 0) {
            sm.ksel = k;
            sm.base = base;
            sm.thr = thr;
            sm.total = total;
            if (!(total > 0.0)) sm.status = RS_SEQ_UNDERFLOW;
        }
    }
    __syncthreads();
    if (sm.status != RS_SEQ_OK) {
        if (tid == 0) write_outcome(P, row, -1, -1, sm.status);
        zero_residual_row(P, row);
        return;
    }

    // element values of the final distribution (unnormalised, target units)
    const float a_last = (internal && MODE == RS_MODE_RESISPEC) ? sm.st_a[last] : 0.0f;
    auto final_value = [&](float lt, float ld, int j) -> float {
        const float R = exp2_fast(expo(lt, c2h, c2l, Kt));
        if (!internal) return R;
        const float Q = exp2_fast(expo(ld, c2h, c2l, Kd));
        float A, Bv;
        chain_terms<MODE, true>(R, Q, j, sm, last, A, Bv);
        if (MODE == RS_MODE_SPECINFER) return A;
        return fmaf(a_last, Bv - A, A);
    };

    const int tile_elems = ti * ITER;
    const int CH = tile_elems / kBlock;           // contiguous elements per thread
    const int t0 = sm.ksel * tile_elems + tid * CH;
    double own = 0.0;
    for (int c = 0; c < CH; c += VEC) {
        float tv[VEC], dv[VEC];
        load_vec<In, VEC>(tg, t0 + c, V, tv);
        if (internal) load_vec<In, VEC>(dg, t0 + c, V, dv);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            const int j = t0 + c + e;
            if (j < V) own += (double)final_value(tv[e], internal ? dv[e] : 0.0f, j);
        }
    }
    // block exclusive scan of `own`
    const double incl = wave_incl_scan(own, lane);
    if (lane == 63) sm.scan_w[wid] = incl;
    __syncthreads();
    double wbase = 0.0;
    for (int w = 0; w < wid; ++w) wbase += sm.scan_w[w];
    const double excl = wbase + incl - own;
    const double thr = sm.thr;
    const double tbase = sm.base;
    const bool cond = (own > 0.0) && (tbase + excl + own > thr);
    const uint64_t cmask = __ballot(cond);
    if (lane == 0) sm.first_w[wid] = cmask ? wid * 64 + (__ffsll((unsigned long long)cmask) - 1) : kBlock;
    __syncthreads();
    if (tid == 0) {
        int first = kBlock;
        for (int w = 0; w < kWaves; ++w) first = min(first, sm.first_w[w]);
        sm.first_w[0] = first;
        sm.token = -1;
    }
    __syncthreads();
    int chosen = sm.first_w[0];
    bool fallback = false;
    if (chosen == kBlock) {   // rounding guard: last thread of the tile with mass
        const uint64_t pm = __ballot(own > 0.0);
        if (lane == 0) sm.first_w[1 + wid] = pm ? wid * 64 + (63 - __clzll((long long)pm)) : -1;
        __syncthreads();
        if (tid == 0) {
            int lastt = -1;
            for (int w = 0; w < kWaves; ++w) lastt = max(lastt, sm.first_w[1 + w]);
            sm.first_w[0] = lastt;
        }
        __syncthreads();
        chosen = sm.first_w[0];
        fallback = true;
    }
    if (tid == chosen) {
        double acc = tbase + excl;
        int tok = -1, lastpos = -1;
        for (int c = 0; c < CH && tok < 0; c += VEC) {
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
        if (tok < 0) tok = lastpos;
        sm.token = tok;
    }
    __syncthreads();
    const int32_t tok = sm.token;
    if (tid == 0) {
        if (tok < 0) write_outcome(P, row, -1, -1, RS_SEQ_UNDERFLOW);
        else write_outcome(P, row, -1, tok, RS_SEQ_OK);
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

// ----------------------------------------------------------- walk kernel ----

__global__ void rs_walk_kernel(const int32_t* __restrict__ node_child,
                               const int32_t* __restrict__ node_tok,
                               const int32_t* __restrict__ node_status,
                               const int32_t* __restrict__ node_token, int32_t B, int32_t N,
                               int32_t max_depth, int32_t* __restrict__ out_tokens,
                               int32_t* __restrict__ out_len, int32_t* __restrict__ out_status) {
    const int32_t b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    const int64_t W = (int64_t)max_depth + 1;
    int32_t* out = out_tokens + (int64_t)b * W;
    const int64_t base = (int64_t)b * N;
    for (int64_t i = 0; i < W; ++i) out[i] = -1;
    int32_t n = 0, len = 0, status = RS_SEQ_OK;
    for (int32_t steps = 0; steps <= N; ++steps) {
        const int32_t st = node_status[base + n];
        if (st != RS_SEQ_OK) {
            status = st;
            break;
        }
        const int32_t c = node_child[base + n];
        if (c >= 0) {
            if (c <= n || c >= N) {
                status = RS_SEQ_BAD_TREE;
                break;
            }
            if (len >= max_depth) {
                status = RS_SEQ_DEPTH_EXCEEDED;
                break;
            }
            out[len++] = node_token[base + c];
            n = c;
            continue;
        }
        const int32_t t = node_tok[base + n];
        if (t >= 0) out[len] = t;
        break;
    }
    if (status != RS_SEQ_OK) {
        for (int64_t i = 0; i < W; ++i) out[i] = -1;
        len = -1;
    }
    out_len[b] = len;
    if (out_status) out_status[b] = status;
}

}  // namespace

// ================================================================ host ABI ====

namespace {

constexpr int kWalkBlock = 256;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

rs_status check_params(const rs_params* prm) {
    if (!prm) return RS_ERR_INVALID_ARG;
    if (prm->mode != RS_MODE_RESISPEC && prm->mode != RS_MODE_SPECINFER) return RS_ERR_INVALID_ARG;
    if (prm->logits_dtype != RS_F32 && prm->logits_dtype != RS_BF16) return RS_ERR_INVALID_ARG;
    if (!(prm->temperature > 0.0f) || !std::isfinite(prm->temperature)) return RS_ERR_INVALID_ARG;
    return RS_OK;
}

template <typename In, int VEC, int UNR, int MODE>
hipError_t launch_rows_t(KParams P, int64_t nrows, hipStream_t s) {
    constexpr int64_t ITER = (int64_t)kBlock * VEC * UNR;
    const int64_t niters = ((int64_t)P.V + ITER - 1) / ITER;
    const int64_t tile_iters = (niters + kMaxTiles - 1) / kMaxTiles;
    P.niters = (int32_t)niters;
    P.tile_iters = (int32_t)tile_iters;
    P.ntiles = (int32_t)((niters + tile_iters - 1) / tile_iters);
    hipLaunchKernelGGL((rs_row_kernel<In, VEC, UNR, MODE>), dim3((unsigned)nrows), dim3(kBlock), 0, s, P);
    return hipGetLastError();
}

template <int MODE>
hipError_t launch_rows_m(const KParams& P, int dtype, bool vec, int64_t nrows, hipStream_t s) {
    if (dtype == RS_BF16) {
        return vec ? launch_rows_t<uint16_t, 8, 2, MODE>(P, nrows, s)
                   : launch_rows_t<uint16_t, 1, 4, MODE>(P, nrows, s);
    }
    return vec ? launch_rows_t<float, 4, 2, MODE>(P, nrows, s)
               : launch_rows_t<float, 1, 4, MODE>(P, nrows, s);
}

hipError_t launch_rows(const KParams& P, const rs_params* prm, bool vec, int64_t nrows, hipStream_t s) {
    if (prm->mode == RS_MODE_SPECINFER) return launch_rows_m<RS_MODE_SPECINFER>(P, prm->logits_dtype, vec, nrows, s);
    return launch_rows_m<RS_MODE_RESISPEC>(P, prm->logits_dtype, vec, nrows, s);
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
    // c2 = c2h + c2l with c2h strictly below c2, so c2l > 0: then a -inf logit gives
    // the exponent -inf (never -inf + inf) and contributes exactly zero.
    const double c2 = 1.4426950408889634 / (double)prm->temperature;
    float c2h = (float)c2;
    if ((double)c2h >= c2) c2h = std::nextafter(c2h, 0.0f);
    P.c2h = c2h;
    P.c2l = (float)(c2 - (double)c2h);
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
    hipLaunchKernelGGL(rs_walk_kernel, dim3((unsigned)((B + kWalkBlock - 1) / kWalkBlock)),
                       dim3(kWalkBlock), 0, s, node_child, node_tok, node_status, node_token, B, N,
                       max_depth, out_tokens, out_len, out_status);
    return hipGetLastError();
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
