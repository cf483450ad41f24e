// resispec.hip -- gfx950 kernels and C ABI of the ResiSpec verification step.
//
// Paper: "ResiSpec: Enhancing Multi-Candidate Speculative Sampling via Residual
// Distribution Shaping".  One workgroup verifies one tree node (one logits row):
//
//   pass 1   online softmax statistics (max, sum of exp) of the target row and, for
//            nodes with children, the draft row (Preliminary; temperature T);
//   tests    candidate i is accepted iff u_i < R_i(x_i) / D_i(x_i) (Eq. 2 and
//            Algorithm 1), evaluated in fp64 on gathered logits;
//   pass i+1 after the i-th rejection one more pass over the row computes the sums the
//            residual update needs:
//              standard (Eq. 1/2):   S = sum_j max(R_j - D_j, 0)
//              ResiSpec (Algorithm 1, GetProxy): M = sum_{j != x0} min(Z D_j, R_j) and
//                                    SR = sum_{j != x0} R_j, with Z = D(x0) - R(x0).
//            GetProxy's one-shot redistribution of Delta = Z - M into the capacity
//            R_j - m_j gives, with a = Delta / (SR - M), the residual
//              R'_j = ((1 - a) min(Z D_j, R_j) + a R_j) / Z   (j != x0),   R'_x0 = 0,
//            i.e. norm(max(R - K, 0)) for the proxy K = R - r, K(x0) = D(x0).  So the
//            residual is never materialised: every pass re-derives R_j from (p_j, q_j)
//            through the chain of per-rejection scalars;
//   draw     when every candidate is rejected (or the node is a leaf: bonus draw from
//            p), the token is the smallest j whose running sum of the final residual in
//            vocabulary order exceeds u * total.  The last pass records per-tile partial
//            sums, so the draw re-reads a single tile.
//
// Precision: elements in fp32 (bf16 widened exactly), every sum accumulated in fp64,
// the per-candidate probabilities and the scalar chain in fp64.
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
constexpr float kLog2e = 1.4426950408889634f;

// ------------------------------------------------------------------ loads ----

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float widen(float x) { return x; }
__device__ __forceinline__ float widen(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// VEC consecutive elements starting at element idx; elements at or beyond V read as
// -inf, which makes them contribute exactly zero to every sum below.
template <typename In, int VEC>
struct Loader;

template <>
struct Loader<float, 4> {
    static __device__ __forceinline__ void load(const float* __restrict__ row, int64_t idx,
                                                int64_t V, float (&v)[4]) {
        if (idx < V) {
            const float4 t = *reinterpret_cast<const float4*>(row + idx);
            v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = -INFINITY;
        }
    }
};

template <>
struct Loader<uint16_t, 8> {
    static __device__ __forceinline__ void load(const uint16_t* __restrict__ row, int64_t idx,
                                                int64_t V, float (&v)[8]) {
        if (idx < V) {
            const uint4 t = *reinterpret_cast<const uint4*>(row + idx);
            v[0] = bf16_lo(t.x); v[1] = bf16_hi(t.x);
            v[2] = bf16_lo(t.y); v[3] = bf16_hi(t.y);
            v[4] = bf16_lo(t.z); v[5] = bf16_hi(t.z);
            v[6] = bf16_lo(t.w); v[7] = bf16_hi(t.w);
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = -INFINITY;
        }
    }
};

template <typename In>
struct Loader<In, 1> {
    static __device__ __forceinline__ void load(const In* __restrict__ row, int64_t idx,
                                                int64_t V, float (&v)[1]) {
        v[0] = (idx < V) ? widen(row[idx]) : -INFINITY;
    }
};

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

struct StepConst {      // one rejection, in the order the candidates were tested
    int32_t x;          // rejected token
    float zf, af, invf; // ResiSpec: Z, a, 1/Z.  Standard: invf = 1/S
    float dscalef;      // draft scale of this step (without replacement)
    double z, a, inv, dscale;
};

struct Smem {
    int32_t status;
    int32_t nc;
    int32_t decision;     // -1 continue, >= 0 accepted candidate, -2 fault
    int32_t nrej;
    float ur;
    float mt, md;         // raw-logit row maxima
    double St, Sd;        // sums of exp((l - max)/T)
    int32_t cand_tok[kMaxCand];
    int32_t cand_node[kMaxCand];
    float cand_u[kMaxCand];
    double cand_p[kMaxCand];
    double cand_q[kMaxCand];
    StepConst step[kMaxCand + 1];
    // per-tile partials written by one wave each
    double tpA[kMaxTiles][kWaves];
    double tpB[kMaxTiles][kWaves];
    float tpM[kMaxTiles][kWaves];
    double tileT[kMaxTiles];
    // cross-wave reductions
    float redf[2][kWaves];
    double redd[2][kWaves];
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
    int64_t V;
    float T;
    float c2;          // log2(e) / T
    int32_t worep, bonus, flat;
    int32_t tile_iters; // loop iterations per tile
    int32_t ntiles;
};

// Per-element state of the residual chain after `nsteps` rejections, starting from
// p_j = exp2((lt - mt) c2) / St and q_j likewise (fp32).
template <int MODE>
__device__ __forceinline__ void apply_chain(float& R, float& D, bool& removed, int64_t j,
                                            float q, const StepConst* __restrict__ st,
                                            int nsteps, bool worep) {
    for (int t = 0; t < nsteps; ++t) {
        const StepConst& s = st[t];
        const float Dt = removed ? 0.0f : q * s.dscalef;
        if (MODE == RS_MODE_SPECINFER) {
            R = fmaxf(R - Dt, 0.0f) * s.invf;
        } else {
            if (j == (int64_t)s.x) {
                R = 0.0f;
            } else {
                const float m = fminf(s.zf * Dt, R);
                R = ((1.0f - s.af) * m + s.af * R) * s.invf;
            }
        }
        if (worep && j == (int64_t)s.x) removed = true;
    }
    D = removed ? 0.0f : q * st[nsteps].dscalef;
}

// Quantities of rejection step `i` for one element (chain over steps 0..i-1 first):
//   standard: A = max(R - D, 0), B unused
//   ResiSpec: A = min(Z D, R), B = R, both zero at the rejected token.
template <int MODE>
__device__ __forceinline__ void step_terms(float lt, float ld, int64_t j, const Smem& sm, float c2,
                                           float invSt, float invSd, int i, bool worep,
                                           float& A, float& Bv) {
    const float p = exp2f((lt - sm.mt) * c2) * invSt;
    const float q = exp2f((ld - sm.md) * c2) * invSd;
    float R = p, D;
    bool removed = false;
    apply_chain<MODE>(R, D, removed, j, q, sm.step, i, worep);
    if (MODE == RS_MODE_SPECINFER) {
        A = fmaxf(R - D, 0.0f);
        Bv = 0.0f;
    } else {
        const bool x0 = (j == (int64_t)sm.step[i].x);
        A = x0 ? 0.0f : fminf(sm.step[i].zf * D, R);
        Bv = x0 ? 0.0f : R;
    }
}

// Scalar chain for the accept test of candidate i (fp64).
template <int MODE>
__device__ double scalar_residual(const Smem& sm, int i, double p, double q, int32_t x,
                                  bool worep, double& Dout) {
    double R = p;
    bool removed = false;
    for (int t = 0; t < i; ++t) {
        const StepConst& s = sm.step[t];
        const double Dt = removed ? 0.0 : q * s.dscale;
        if (MODE == RS_MODE_SPECINFER) {
            const double w = R - Dt;
            R = (w > 0.0 ? w : 0.0) * s.inv;
        } else {
            if (x == s.x) {
                R = 0.0;
            } else {
                const double zd = s.z * Dt;
                const double m = zd < R ? zd : R;
                R = ((1.0 - s.a) * m + s.a * R) / s.z;
            }
        }
        if (worep && x == s.x) removed = true;
    }
    Dout = removed ? 0.0 : q * sm.step[i].dscale;
    return R;
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

template <typename In, int VEC>
__device__ void zero_residual_row(const KParams& P, int64_t row) {
    if (!P.residual_out) return;
    float* out = P.residual_out + row * P.V;
    for (int64_t j = threadIdx.x; j < P.V; j += kBlock) out[j] = 0.0f;
}

// ------------------------------------------------------------ row kernel ----

template <typename In, int VEC, int UNR, int MODE>
__global__ void __launch_bounds__(kBlock) rs_row_kernel(const KParams P) {
    __shared__ Smem sm;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int64_t V = P.V;
    constexpr int64_t ITER = (int64_t)kBlock * VEC * UNR;

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

    // ---- row description: candidates, their uniforms, structural checks
    if (tid == 0) {
        sm.status = RS_SEQ_OK;
        sm.nc = 0;
        sm.decision = -1;
        sm.nrej = 0;
    }
    __syncthreads();
    if (P.flat) {
        if (tid < P.k) {
            sm.cand_tok[tid] = P.cand_ids[row * P.k + tid];
            sm.cand_u[tid] = P.ua_flat[row * P.k + tid];
            sm.cand_node[tid] = tid;
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
                        sm.cand_tok[idx] = P.node_token[(int64_t)b * P.N + m];
                        sm.cand_u[idx] = P.ua[(int64_t)b * P.N + m];
                        sm.cand_node[idx] = m;
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
        zero_residual_row<In, VEC>(P, row);
        return;
    }
    if (nc == 0 && !P.flat && !P.bonus) {
        if (tid == 0) write_outcome(P, row, -1, -1, RS_SEQ_OK);
        zero_residual_row<In, VEC>(P, row);
        return;
    }

    const bool internal = nc > 0;
    const In* __restrict__ tg = reinterpret_cast<const In*>(P.tgt) + row * V;
    const In* __restrict__ dg = reinterpret_cast<const In*>(P.dft) + row * V;
    const float c2 = P.c2;
    const double c2d = (double)kLog2e / (double)P.T;
    const int tile_iters = P.tile_iters;

    // ---- pass 1: softmax statistics (per-lane running max, rescaled sums)
    {
        float mt = -FLT_MAX, md = -FLT_MAX;
        double st = 0.0, sd = 0.0;
        float stile = 0.0f;   // leaf rows: this tile's share of st (same reference mt)
        int64_t it = 0;
        for (int64_t base = 0; base < V; base += ITER, ++it) {
            float tv[UNR][VEC], dv[UNR][VEC];
#pragma unroll
            for (int u = 0; u < UNR; ++u)
                Loader<In, VEC>::load(tg, base + ((int64_t)u * kBlock + tid) * VEC, V, tv[u]);
            if (internal) {
#pragma unroll
                for (int u = 0; u < UNR; ++u)
                    Loader<In, VEC>::load(dg, base + ((int64_t)u * kBlock + tid) * VEC, V, dv[u]);
            }
            float mx = -FLT_MAX;
#pragma unroll
            for (int u = 0; u < UNR; ++u)
#pragma unroll
                for (int e = 0; e < VEC; ++e) mx = fmaxf(mx, tv[u][e]);
            if (mx > mt) {
                const double f = exp2(((double)mt - (double)mx) * c2d);
                st *= f;
                stile = (float)(stile * f);
                mt = mx;
            }
            float acc = 0.0f;
#pragma unroll
            for (int u = 0; u < UNR; ++u)
#pragma unroll
                for (int e = 0; e < VEC; ++e) acc += exp2f((tv[u][e] - mt) * c2);
            st += (double)acc;
            stile += acc;
            if (internal) {
                float my = -FLT_MAX;
#pragma unroll
                for (int u = 0; u < UNR; ++u)
#pragma unroll
                    for (int e = 0; e < VEC; ++e) my = fmaxf(my, dv[u][e]);
                if (my > md) {
                    sd *= exp2(((double)md - (double)my) * c2d);
                    md = my;
                }
                float accd = 0.0f;
#pragma unroll
                for (int u = 0; u < UNR; ++u)
#pragma unroll
                    for (int e = 0; e < VEC; ++e) accd += exp2f((dv[u][e] - md) * c2);
                sd += (double)accd;
            } else {
                const bool tile_end = ((it + 1) % tile_iters == 0) || (base + ITER >= V);
                if (tile_end) {
                    const int tile = (int)(it / tile_iters);
                    const float mw = wave_max(mt);
                    const double sw = wave_sum((double)stile * exp2(((double)mt - (double)mw) * c2d));
                    if (lane == 0) {
                        sm.tpM[tile][wid] = mw;
                        sm.tpA[tile][wid] = sw;
                    }
                    stile = 0.0f;
                }
            }
        }
        // block combine
        const float mwt = wave_max(mt);
        const double swt = wave_sum(st * exp2(((double)mt - (double)mwt) * c2d));
        float mwd = -FLT_MAX;
        double swd = 0.0;
        if (internal) {
            mwd = wave_max(md);
            swd = wave_sum(sd * exp2(((double)md - (double)mwd) * c2d));
        }
        if (lane == 0) {
            sm.redf[0][wid] = mwt;
            sm.redd[0][wid] = swt;
            sm.redf[1][wid] = mwd;
            sm.redd[1][wid] = swd;
        }
        __syncthreads();
        if (tid == 0) {
            float m0 = -FLT_MAX, m1 = -FLT_MAX;
            for (int w = 0; w < kWaves; ++w) {
                m0 = fmaxf(m0, sm.redf[0][w]);
                m1 = fmaxf(m1, sm.redf[1][w]);
            }
            double s0 = 0.0, s1 = 0.0;
            for (int w = 0; w < kWaves; ++w) {
                s0 += sm.redd[0][w] * exp2(((double)sm.redf[0][w] - (double)m0) * c2d);
                if (internal) s1 += sm.redd[1][w] * exp2(((double)sm.redf[1][w] - (double)m1) * c2d);
            }
            sm.mt = m0;
            sm.md = m1;
            sm.St = s0;
            sm.Sd = s1;
            if (!(s0 > 0.0) || (internal && !(s1 > 0.0))) sm.status = RS_SEQ_UNDERFLOW;
            sm.step[0].dscale = 1.0;
            sm.step[0].dscalef = 1.0f;
        }
        __syncthreads();
        if (sm.status != RS_SEQ_OK) {
            if (tid == 0) write_outcome(P, row, -1, -1, sm.status);
            zero_residual_row<In, VEC>(P, row);
            return;
        }
    }

    // ---- candidate probabilities in fp64 (gathers)
    if (tid < nc) {
        const int32_t x = sm.cand_tok[tid];
        double pc = 0.0, qc = 0.0;
        if (x >= 0 && (int64_t)x < V) {
            const double T = (double)P.T;
            pc = exp(((double)widen(tg[x]) - (double)sm.mt) / T) / sm.St;
            qc = exp(((double)widen(dg[x]) - (double)sm.md) / T) / sm.Sd;
        }
        sm.cand_p[tid] = pc;
        sm.cand_q[tid] = qc;
    }
    __syncthreads();

    const float invSt = (float)(1.0 / sm.St);
    const float invSd = internal ? (float)(1.0 / sm.Sd) : 0.0f;
    const bool worep = P.worep != 0;

    // ---- sequential accept / reject
    int i = 0;
    for (; i < nc; ++i) {
        if (tid == 0) {
            const int32_t x = sm.cand_tok[i];
            const float u = sm.cand_u[i];
            int dec = -1;
            if (x < 0 || (int64_t)x >= V) {
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
                    StepConst& s = sm.step[i];
                    s.x = x;
                    s.z = Dx - Rx;   // ResiSpec budget; unused by the standard update
                    s.zf = (float)s.z;
                }
            }
            sm.decision = dec;
        }
        __syncthreads();
        if (sm.decision != -1) break;

        // rejection pass: sums of step i with per-tile partials
        {
            double accA = 0.0, accB = 0.0;   // this tile's lane partials
            int64_t it = 0;
            for (int64_t base = 0; base < V; base += ITER, ++it) {
                float tv[UNR][VEC], dv[UNR][VEC];
#pragma unroll
                for (int u = 0; u < UNR; ++u) {
                    Loader<In, VEC>::load(tg, base + ((int64_t)u * kBlock + tid) * VEC, V, tv[u]);
                    Loader<In, VEC>::load(dg, base + ((int64_t)u * kBlock + tid) * VEC, V, dv[u]);
                }
                float fa = 0.0f, fb = 0.0f;
#pragma unroll
                for (int u = 0; u < UNR; ++u) {
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        const int64_t j = base + ((int64_t)u * kBlock + tid) * VEC + e;
                        float A, Bv;
                        step_terms<MODE>(tv[u][e], dv[u][e], j, sm, c2, invSt, invSd, i, worep, A, Bv);
                        fa += A;
                        fb += Bv;
                    }
                }
                accA += (double)fa;
                accB += (double)fb;
                const bool tile_end = ((it + 1) % tile_iters == 0) || (base + ITER >= V);
                if (tile_end) {
                    const int tile = (int)(it / tile_iters);
                    const double wa = wave_sum(accA);
                    const double wb = (MODE == RS_MODE_RESISPEC) ? wave_sum(accB) : 0.0;
                    if (lane == 0) {
                        sm.tpA[tile][wid] = wa;
                        sm.tpB[tile][wid] = wb;
                    }
                    accA = accB = 0.0;
                }
            }
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
            const double totA = __shfl(wave_sum(A), 0, 64);
            const double totB = __shfl(wave_sum(Bv), 0, 64);
            const double z = sm.step[i].z;
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
                StepConst& s = sm.step[i];
                if (MODE == RS_MODE_SPECINFER && !(totA > 0.0)) {
                    sm.status = RS_SEQ_UNDERFLOW;
                    sm.decision = -2;
                }
                s.a = a;
                s.af = (float)a;
                s.inv = inv;
                s.invf = (float)inv;
                StepConst& nx = sm.step[i + 1];
                if (worep) {
                    const double rest = 1.0 - sm.cand_q[i] * s.dscale;
                    nx.dscale = rest > 0.0 ? s.dscale / rest : 0.0;
                } else {
                    nx.dscale = 1.0;
                }
                nx.dscalef = (float)nx.dscale;
                sm.nrej = i + 1;
            }
        }
        __syncthreads();
        if (sm.decision == -2) break;
    }

    if (sm.decision == -2) {
        if (tid == 0) write_outcome(P, row, -1, -1, sm.status);
        zero_residual_row<In, VEC>(P, row);
        return;
    }
    if (sm.decision >= 0) {
        if (tid == 0) {
            const int d = sm.decision;
            write_outcome(P, row, sm.cand_node[d], sm.cand_tok[d], RS_SEQ_OK);
        }
        zero_residual_row<In, VEC>(P, row);
        return;
    }

    // ---- every candidate rejected, or no candidates: inverse-CDF draw
    const float u = sm.ur;
    if (!(u >= 0.0f && u < 1.0f)) {
        if (tid == 0) write_outcome(P, row, -1, -1, RS_SEQ_BAD_UNIFORM);
        zero_residual_row<In, VEC>(P, row);
        return;
    }
    const int last = nc - 1;   // index of the last rejection step (internal rows)
    if (wid == 0) {
        double T = 0.0;
        if (lane < P.ntiles) {
            if (internal) {
                T = sm.tileT[lane];
            } else {
                for (int w = 0; w < kWaves; ++w)
                    T += sm.tpA[lane][w] * exp2(((double)sm.tpM[lane][w] - (double)sm.mt) * c2d);
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
        zero_residual_row<In, VEC>(P, row);
        return;
    }

    // element values of the final distribution (unnormalised)
    const double a_last = (internal && MODE == RS_MODE_RESISPEC) ? sm.step[last].a : 0.0;
    auto final_value = [&](float lt, float ld, int64_t j) -> float {
        if (!internal) return exp2f((lt - sm.mt) * c2);
        float A, Bv;
        step_terms<MODE>(lt, ld, j, sm, c2, invSt, invSd, last, worep, A, Bv);
        if (MODE == RS_MODE_SPECINFER) return A;
        const float af = (float)a_last;
        return (1.0f - af) * A + af * Bv;
    };

    const int64_t tile_elems = (int64_t)tile_iters * ITER;
    const int64_t CH = tile_elems / kBlock;           // contiguous elements per thread
    const int64_t t0 = (int64_t)sm.ksel * tile_elems + (int64_t)tid * CH;
    double own = 0.0;
    for (int64_t c = 0; c < CH; c += VEC) {
        float tv[VEC], dv[VEC];
        Loader<In, VEC>::load(tg, t0 + c, V, tv);
        if (internal) Loader<In, VEC>::load(dg, t0 + c, V, dv);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            const int64_t j = t0 + c + e;
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
        int64_t tok = -1, lastpos = -1;
        for (int64_t c = 0; c < CH && tok < 0; c += VEC) {
            float tv[VEC], dv[VEC];
            Loader<In, VEC>::load(tg, t0 + c, V, tv);
            if (internal) Loader<In, VEC>::load(dg, t0 + c, V, dv);
            for (int e = 0; e < VEC; ++e) {
                const int64_t j = t0 + c + e;
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
        sm.token = (int32_t)tok;
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
        for (int64_t j = tid; j < V; j += kBlock) {
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
    const int64_t niters = (P.V + ITER - 1) / ITER;
    const int64_t tile_iters = (niters + kMaxTiles - 1) / kMaxTiles;
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
    return vec ? launch_rows_t<float, 4, 4, MODE>(P, nrows, s)
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
    P.V = V;
    P.T = prm->temperature;
    P.c2 = (float)(1.4426950408889634 / (double)prm->temperature);
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
