// draft.hip -- the draft step on gfx950: the candidate tokens of every node's children
// drawn from the node's draft row, and every node's uniforms, ahead of verification
// (resispec.hip).  Declared in resispec.h (resispec_draft_candidates).

#include "common.h"

namespace {

// The step before verification: every node's uniforms and the candidate tokens of
// every node's children, drawn on the device.  Uniforms come from Philox4x32-10
// (Salmon, Moraes, Dror and Shaw, SC'11): node n of sequence b takes counter
// (n, b, offset low, offset high) under key (seed low, seed high); word 0 is its
// u_accept, word 1 its u_resample and word 2 the uniform that draws the node's own
// token from its parent's draft distribution.  Candidates are inverse-CDF draws in
// vocabulary order from softmax(draft / T) (children in ascending node index); without
// replacement each draw removes its token from the distribution before the next.

__device__ __forceinline__ void philox4x32_10(uint32_t (&c)[4], uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint32_t lo0 = 0xD2511F53u * c[0], hi0 = __umulhi(0xD2511F53u, c[0]);
        const uint32_t lo1 = 0xCD9E8D57u * c[2], hi1 = __umulhi(0xCD9E8D57u, c[2]);
        const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0;
        c[1] = lo1;
        c[2] = n2;
        c[3] = lo0;
    }
}

__device__ __forceinline__ float u01(uint32_t w) { return (float)(w >> 8) * (1.0f / 16777216.0f); }

struct DParams {
    const void* dft;
    const int32_t* parent;
    int32_t* node_token;
    float* ua;
    float* ur;
    int32_t* out_status;   // per sequence, may be NULL
    int32_t B, N, V;
    float c2h, c2l;
    int32_t worep;
    uint32_t seed_lo, seed_hi, off_lo, off_hi;
    int32_t G, nslots;
};

// The draft kernel's shared state: one fp64 total per slot (the wave that sweeps a slot
// sums its lanes' partials itself), so about 2 KB instead of the verification kernels'
// 77 KB.  While a row's draws leave one wave running (draws without replacement, or a
// single child), the other waves' registers and the small LDS let further rows'
// workgroups start on the CU and stream.
struct DraftSmem {
    int32_t decision;
    int32_t next_slot;
    double total;
    int32_t wcount[kMaxWaves];
    int32_t wbad[kMaxWaves];
    int32_t cand_tok[kMaxCand];
    int32_t cand_node[kMaxCand];
    float cand_u[kMaxCand];
    float wmax[2][kMaxWaves];
    double slotA[kMaxSlots];
};

// Four waves per row workgroup (the verification kernels take eight): a row's draws
// without replacement keep one wave busy after the pass, and a smaller workgroup lets a
// further row start streaming in the wave slots the others free (serving workload:
// 0.302 -> 0.240 ms against eight waves).
constexpr int kDraftBlock = 256;

template <typename In, int VEC, int UNR>
__global__ void __launch_bounds__(kDraftBlock) __attribute__((amdgpu_waves_per_eu(4))) rs_draft_kernel(const DParams P) {
    constexpr int kBlock = kDraftBlock;
    __shared__ DraftSmem sm;
    constexpr int kWaves = kBlock / 64;
    constexpr int CHUNK = 64 * VEC * UNR;
    using W = Vec<In, VEC>;
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int V = P.V, G = P.G, nslots = P.nslots;
    const int32_t g = blockIdx.x;
    const int32_t n = g / P.B, b = g - n * P.B;
    const int64_t row = (int64_t)b * P.N + n;
    const In* __restrict__ dg = reinterpret_cast<const In*>(P.dft) + row * V;

    if (tid == 0) {
        uint32_t c[4] = {(uint32_t)n, (uint32_t)b, P.off_lo, P.off_hi};
        philox4x32_10(c, P.seed_lo, P.seed_hi);
        P.ua[row] = u01(c[0]);
        P.ur[row] = u01(c[1]);
        if (n == 0) P.node_token[row] = -1;
        sm.next_slot = kWaves;
    }
    // children of node n (ascending node index) and the uniforms that draw them; the
    // draft row is only read when there are children
    const int64_t sb = (int64_t)b * P.N;
    int nc = 0, anybad = 0;
    for (int base = 0; base < P.N; base += kBlock) {
        const int m = base + tid;
        bool holder = false;
        int bad = 0;
        if (m < P.N) {
            const int32_t pm = P.parent[sb + m];
            bad = (m == 0) ? (pm != -1) : (pm < 0 || pm >= m);
            holder = m > n && pm == n;
        }
        const uint64_t cm = __ballot(holder);
        const uint64_t bm = __ballot(bad);
        if (lane == 0) {
            sm.wcount[wid] = __popcll(cm);
            sm.wbad[wid] = bm != 0;
        }
        __syncthreads();
        int rank = nc + __popcll(cm & __lanemask_lt());
        for (int w = 0; w < kWaves; ++w) {
            rank += (w < wid) ? sm.wcount[w] : 0;
            nc += sm.wcount[w];
            anybad |= sm.wbad[w];
        }
        if (holder && rank < kMaxCand) {
            uint32_t c[4] = {(uint32_t)m, (uint32_t)b, P.off_lo, P.off_hi};
            philox4x32_10(c, P.seed_lo, P.seed_hi);
            sm.cand_node[rank] = m;
            sm.cand_u[rank] = u01(c[2]);
        }
        __syncthreads();
    }
    if (n == 0 && tid == 0 && P.out_status) P.out_status[b] = anybad ? RS_SEQ_BAD_TREE : RS_SEQ_OK;
    if (anybad) {
        // a malformed tree: every node's own row marks the node
        if (n > 0 && tid == 0) P.node_token[row] = -1;
        return;
    }
    if (nc > kMaxCand) {
        // too many children to draw: all of them keep token -1
        for (int m = n + 1 + tid; m < P.N; m += kBlock)
            if (P.parent[sb + m] == n) P.node_token[sb + m] = -1;
        return;
    }
    if (nc == 0) return;
    // this wave's first chunk; its maximum fixes the row's exponent reference
    typename W::raw pre[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) pre[u] = W::template load<true>(dg, wid * G * CHUNK + lane * VEC + u * 64 * VEC, V);
    {
        float mx = -FLT_MAX;
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            float v[VEC];
            W::unpack(pre[u], v);
#pragma unroll
            for (int e = 0; e < VEC; ++e) mx = fmaxf(mx, v[e]);
        }
        mx = wave_max(mx);
        if (lane == 0) sm.wmax[0][wid] = mx;
    }
    __syncthreads();
    const float c2h = P.c2h, c2l = P.c2l;

    // ---- one pass: the draft row's sum of exp2 against a fixed reference, per slot
    float K;
    {
        float m0 = -FLT_MAX;
        for (int w = 0; w < kWaves; ++w) m0 = fmaxf(m0, sm.wmax[0][w]);
        K = kref(m0, c2h);
    }
    for (int attempt = 0;; ++attempt) {
        float fa = 0.0f;
        wave_sweep<In, VEC, UNR, false, 1, true>(dg, dg, V, G, nslots, 0, false, pre, pre, &sm.next_slot,
            [&](const float (&t)[UNR][VEC], const float (&)[UNR][VEC], int, int) {
#pragma unroll
                for (int u = 0; u < UNR; ++u)
#pragma unroll
                    for (int e = 0; e < VEC; ++e) fa += exp2_fast(expo(t[u][e], c2h, c2l, K));
            },
            [&](int slot) {
                // the slot's total: its lanes' partials summed in a fixed order, so the
                // total does not depend on which wave swept the slot
                const double v = wave_sum((double)fa);
                if (lane == 0) sm.slotA[slot] = v;
                fa = 0.0f;
            });
        __syncthreads();
        if (wid == 0) {
            double a0 = 0.0;
            for (int s2 = lane; s2 < nslots; s2 += 64) a0 += sm.slotA[s2];
            const double s0 = wave_sum(a0);
            if (lane == 0) {
                sm.total = s0;
                sm.decision = (s0 >= kLowSum && s0 < INFINITY) ? -1 : -3;
                sm.next_slot = kWaves;
            }
        }
        __syncthreads();
        if (sm.decision != -3) break;
        if (attempt == 1) {
            // no usable distribution: the children keep token -1
            if (tid < nc) P.node_token[sb + sm.cand_node[tid]] = -1;
            return;
        }
        float mx = -FLT_MAX;
        wave_sweep<In, VEC, UNR, false, 0, false>(dg, dg, V, G, nslots, 0, false, pre, pre, &sm.next_slot,
            [&](const float (&t)[UNR][VEC], const float (&)[UNR][VEC], int, int) {
#pragma unroll
                for (int u = 0; u < UNR; ++u)
#pragma unroll
                    for (int e = 0; e < VEC; ++e) mx = fmaxf(mx, t[u][e]);
            },
            [](int) {});
        mx = wave_max(mx);
        if (lane == 0) sm.wmax[0][wid] = mx;
        __syncthreads();
        float m0 = -FLT_MAX;
        for (int w = 0; w < kWaves; ++w) m0 = fmaxf(m0, sm.wmax[0][w]);
        K = kref(m0, c2h);
        if (tid == 0) {
            sm.decision = -1;
            sm.next_slot = kWaves;
        }
        __syncthreads();
    }
    // ---- the draws: inverse CDF over the slot totals, then inside one slot.  Draws with
    // replacement are independent and spread over the waves; without replacement each
    // draw depends on the tokens before it and wave 0 takes them in order.
    const bool worep = P.worep != 0;
    if (worep && wid != 0) return;
    const int R = G * VEC * UNR;          // elements of a slot per lane
    // slot totals in vocabulary order, lane l holding slots 4l .. 4l+3.  Without
    // replacement a draw replaces its slot's total by the fp64 sum of the slot's elements
    // that remain (computed in the draw below), so the mass left is always a sum of
    // what remains, never the total less the removed mass.
    double Ts[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int s2 = 4 * lane + q;
        Ts[q] = s2 < nslots ? sm.slotA[s2] : 0.0;
    }
    for (int i = worep ? 0 : wid; i < nc; i += worep ? 1 : kWaves) {
        // removed tokens (lane j holds removed token j, j < i)
        const int32_t rtok = (worep && lane < i) ? sm.cand_tok[lane] : -1;
        const int rslot = rtok >= 0 ? (rtok / CHUNK) / G : -1;
        double own = 0.0;
#pragma unroll
        for (int q = 0; q < 4; ++q) own += Ts[q];
        const double incl = wave_incl_scan(own, lane);
        const double excl = incl - own;
        const double thr = (double)sm.cand_u[i] * readlane_d(incl, 63);
        uint64_t hit = __ballot(own > 0.0 && incl > thr);
        int L = hit ? (__ffsll((unsigned long long)hit) - 1) : -1;
        if (L < 0) {
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
        int32_t tok = -1;
        double tval = 0.0;
        if (ks >= 0) {
            // removed tokens inside slot ks (wave-uniform list, read one by one below)
            const uint64_t rin = __ballot(rtok >= 0 && rslot == ks);
            const int t0 = ks * G * CHUNK + lane * R;
            auto value = [&](float l, int j) -> float {
                float v = exp2_fast(expo(l, c2h, c2l, K));
                uint64_t m = rin;
                while (m) {
                    const int jl = __ffsll((unsigned long long)m) - 1;
                    m &= m - 1;
                    if (j == __builtin_amdgcn_readlane(rtok, jl)) v = 0.0f;
                }
                return v;
            };
            constexpr int kRegRun = 32;
            float vals[kRegRun];
            double own2 = 0.0;
            const bool inreg = R <= kRegRun;
            if (inreg) {
#pragma unroll
                for (int c = 0; c < kRegRun; c += VEC) {
                    float dv[VEC];
                    if (c < R) load_vec<In, VEC>(dg, t0 + c, V, dv);
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        const int j = t0 + c + e;
                        const float v = (c < R && j < V) ? value(dv[e], j) : 0.0f;
                        vals[c + e] = v;
                        own2 += (double)v;
                    }
                }
            } else {
                for (int c = 0; c < R; c += VEC) {
                    float dv[VEC];
                    load_vec<In, VEC>(dg, t0 + c, V, dv);
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        const int j = t0 + c + e;
                        if (j < V) own2 += (double)value(dv[e], j);
                    }
                }
            }
            const double incl2 = wave_incl_scan(own2, lane);
            const double excl2 = incl2 - own2;
            const uint64_t hit2 = __ballot(own2 > 0.0 && base + incl2 > thr);
            int L2 = hit2 ? (__ffsll((unsigned long long)hit2) - 1) : -1;
            const bool fallback = L2 < 0;
            if (fallback) {
                const uint64_t pos = __ballot(own2 > 0.0);
                L2 = pos ? 63 - __clzll((long long)pos) : -1;
            }
            float tv = 0.0f;
            if (lane == L2) {
                double acc = base + excl2;
                int lastpos = -1;
                float lastv = 0.0f;
                if (inreg) {
#pragma unroll
                    for (int c = 0; c < kRegRun; ++c) {
                        const float v = vals[c];
                        const int j = t0 + c;
                        if (tok < 0 && c < R && j < V) {
                            if (v > 0.0f) {
                                lastpos = j;
                                lastv = v;
                            }
                            acc += (double)v;
                            if (!fallback && v > 0.0f && acc > thr) {
                                tok = j;
                                tv = v;
                            }
                        }
                    }
                } else {
                    for (int c = 0; c < R && tok < 0; c += VEC) {
                        float dv[VEC];
                        load_vec<In, VEC>(dg, t0 + c, V, dv);
                        for (int e = 0; e < VEC; ++e) {
                            const int j = t0 + c + e;
                            if (j >= V) break;
                            const float v = value(dv[e], j);
                            if (v > 0.0f) {
                                lastpos = j;
                                lastv = v;
                            }
                            acc += (double)v;
                            if (!fallback && v > 0.0f && acc > thr) {
                                tok = j;
                                tv = v;
                                break;
                            }
                        }
                    }
                }
                if (tok < 0) {
                    tok = lastpos;
                    tv = lastv;
                }
            }
            if (L2 >= 0) {
                tok = __builtin_amdgcn_readlane(tok, L2);
                tval = (double)readlane_f(tv, L2);
            }
            if (worep && tok >= 0) {
                // the slot's remaining mass: its elements summed in fp64 without the
                // removed tokens and without this draw (own2 is exact up to fp64 rounding
                // of fp32 values, so taking the drawn value out cancels nothing)
                const bool mine = tok >= t0 && tok < t0 + R;
                const double rest = wave_sum(own2 - (mine ? tval : 0.0));
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (4 * lane + q == ks) Ts[q] = rest > 0.0 ? rest : 0.0;
            }
        }
        if (lane == 0) {
            P.node_token[sb + sm.cand_node[i]] = tok;
            sm.cand_tok[i] = tok;
        }
        if (tok < 0 && worep) {
            // nothing left to draw from: the remaining children keep token -1
            for (int i2 = i + 1 + lane; i2 < nc; i2 += 64) P.node_token[sb + sm.cand_node[i2]] = -1;
            break;
        }
        __builtin_amdgcn_wave_barrier();
    }
}

template <typename In, int VEC, int UNR>
hipError_t launch_draft_t(DParams P, hipStream_t s) {
    constexpr int64_t CHUNK = 64 * VEC * UNR;
    const int64_t nch = ((int64_t)P.V + CHUNK - 1) / CHUNK;
    const int64_t G = (nch + kMaxSlots - 1) / kMaxSlots;
    P.G = (int32_t)G;
    P.nslots = (int32_t)((nch + G - 1) / G);
    hipLaunchKernelGGL((rs_draft_kernel<In, VEC, UNR>), dim3((unsigned)((int64_t)P.B * P.N)), dim3(kDraftBlock), 0,
                       s, P);
    return hipGetLastError();
}

}  // namespace

extern "C" {

rs_status resispec_draft_candidates(const void* draft_logits, const int32_t* parent, int32_t B,
                                    int32_t N, int32_t V, const rs_params* prm, uint64_t seed,
                                    uint64_t offset, int32_t* node_token, float* u_accept,
                                    float* u_resample, int32_t* out_status, void* stream) {
    const rs_status ps = check_params(prm);
    if (ps != RS_OK) return ps;
    if (B < 0 || N <= 0 || V <= 0) return RS_ERR_INVALID_ARG;
    if (V > RS_MAX_VOCAB) return RS_ERR_UNSUPPORTED;
    if ((int64_t)B * N > 0x7fffffffLL) return RS_ERR_UNSUPPORTED;
    if (B == 0) return RS_OK;
    if (!draft_logits || !parent || !node_token || !u_accept || !u_resample) return RS_ERR_INVALID_ARG;
    DParams P{};
    P.dft = draft_logits;
    P.parent = parent;
    P.node_token = node_token;
    P.ua = u_accept;
    P.ur = u_resample;
    P.out_status = out_status;
    P.B = B;
    P.N = N;
    P.V = V;
    split_c2(prm->temperature, &P.c2h, &P.c2l);
    P.worep = prm->without_replacement ? 1 : 0;
    P.seed_lo = (uint32_t)seed;
    P.seed_hi = (uint32_t)(seed >> 32);
    P.off_lo = (uint32_t)offset;
    P.off_hi = (uint32_t)(offset >> 32);
    const int64_t esz = prm->logits_dtype == RS_BF16 ? 2 : 4;
    const bool vec = ((int64_t)V * esz) % 16 == 0 && aligned16(draft_logits);
    const hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    if (prm->logits_dtype == RS_BF16)
        e = vec ? launch_draft_t<uint16_t, 8, kUnr16>(P, s) : launch_draft_t<uint16_t, 1, 4>(P, s);
    else
        e = vec ? launch_draft_t<float, 4, kUnr32>(P, s) : launch_draft_t<float, 1, 4>(P, s);
    return e == hipSuccess ? RS_OK : RS_ERR_HIP;
}

}  // extern "C"
