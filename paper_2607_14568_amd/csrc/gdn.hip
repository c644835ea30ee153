// libgdn: gated delta-rule prefill and decode for MI355X (gfx950).
//
// The method (paper, section 2.2 and section 3.2): per head, a state
// S in R^{dv x dk} follows
//     S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T,  o_t = S_t (scale q_t).
// Prefill evaluates it chunk by chunk (section 3.2).  For a chunk of n <= 64
// tokens entering with state S0, with G = cumsum(g), gamma = exp(G),
// Gamma_ri = exp(G_r - G_i) (i <= r), D = diag(exp(G_n - G_r)):
//     A  = strict_lower(diag(beta) (K K^T o Gamma))         token-token product
//     T  = (I + A)^{-1}                                     forward substitution
//     P  = lower(Q K^T o Gamma)                             token-token product
//     U  = T diag(beta) (V - diag(gamma) K S0^T)            per-chunk correction
//     O  = scale (diag(gamma) Q S0^T + P U)                 chunk output
//     S  = gamma_n S0 + U^T D K                             inter-chunk recurrence
// The prefix sums G are formed in fp64: with very negative g (alpha underflowing)
// |G| grows far beyond the range where fp32 differences G_r - G_i keep their
// precision, while every exp() taken of them stays meaningful.
// T, P and the decay vectors depend only on the chunk's own inputs, so they are formed for all
// (chunk, head) pairs at once by k_chunk_terms; k_state_chain then walks the
// chunks of each (sequence, head, 16-row slice of the state) in order, with all
// contractions on MFMA (bf16 operands with fp32 accumulation for bf16 io, fp32
// MFMA for fp32 io) and the state kept in fp32.
//
// Decode (k_decode_step) is the recurrence at T = 1: one pass over the state,
// row by row (rows of S never mix).
#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "gdn.h"

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short short8 __attribute__((ext_vector_type(8)));
typedef uint16_t bf16_t;

constexpr int CH = 64;    // chunk length (tokens)
constexpr int NT = 256;   // threads per workgroup: 4 waves of 64
constexpr int SL = 16;    // state rows (value channels) per chain workgroup

// ------------------------------------------------------------------ conversions
__device__ __forceinline__ float to_f(float x) { return x; }
__device__ __forceinline__ float to_f(bf16_t x) { return __uint_as_float((uint32_t)x << 16); }

template <typename IO> __device__ __forceinline__ IO from_f(float f);
template <> __device__ __forceinline__ float from_f<float>(float f) { return f; }
template <> __device__ __forceinline__ bf16_t from_f<bf16_t>(float f) {
    // round to nearest even; NaN stays NaN
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (bf16_t)(u >> 16);
}

// ------------------------------------------------------------------ MFMA 16x16
// Output layout of both instructions: lane l holds D[4*(l/16) + e][l % 16], e = 0..3.
// Operand layout: lane l feeds row (A) / column (B) l % 16 and KL contraction
// elements; which contraction indices a lane's elements stand for is a free
// choice as long as A and B agree.  Here element e of lane group lg = l/16 in
// step kk is contraction index kk*KS + lg*KL + e.
template <typename IO> struct Mma;

template <> struct Mma<bf16_t> {
    static constexpr int KS = 32;  // contraction length per instruction
    static constexpr int KL = 8;   // contraction elements per lane
    typedef bf16x8 frag;
    __device__ static __forceinline__ floatx4 mma(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    __device__ static __forceinline__ frag load(const bf16_t* p) {   // 16-byte aligned
        return __builtin_bit_cast(frag, *reinterpret_cast<const short8*>(p));
    }
    __device__ static __forceinline__ frag pack(const float* x) {
        short8 s;
#pragma unroll
        for (int e = 0; e < 8; ++e) s[e] = (short)from_f<bf16_t>(x[e]);
        return __builtin_bit_cast(frag, s);
    }
};

template <> struct Mma<float> {
    static constexpr int KS = 4;
    static constexpr int KL = 1;
    typedef float frag;
    __device__ static __forceinline__ floatx4 mma(frag a, frag b, floatx4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    __device__ static __forceinline__ frag load(const float* p) { return *p; }
    __device__ static __forceinline__ frag pack(const float* x) { return x[0]; }
};

// ------------------------------------------------------------------ parameters
struct Params {
    const void* q;
    const void* k;
    const void* v;
    const float* g;
    const float* beta;
    const float* S0;
    void* o;
    float* ST;
    int B, T, H, DV;
    int n_seq;         // dense: B; ragged: number of packed sequences
    int ragged;
    int NC;            // dense: chunks per sequence
    const int32_t* cu; // ragged: raw offsets (device)
    int32_t* seq_start;
    int32_t* seq_len;
    int32_t* chunk_off;  // [n_seq + 1], first chunk slot of each sequence
    float* wsG;          // [slot][H][128]: gamma_r = exp(G_r), then exp(G_n - G_r)
    void* wsT;           // [slot][H][64][64] io type
    void* wsP;           // [slot][H][64][64] io type
    float scale;
};

__device__ __forceinline__ void seq_info(const Params& p, int s, long& start, int& len, int& cbase) {
    if (p.ragged) {
        start = p.seq_start[s];
        len = p.seq_len[s];
        cbase = p.chunk_off[s];
    } else {
        start = (long)s * p.T;
        len = p.T;
        cbase = s * p.NC;
    }
}

// Sanitises the ragged offsets into a nondecreasing partition of [0, T] and
// lays out one workspace slot per chunk of every sequence.
__global__ void k_ragged_setup(const int32_t* cu, int n_seq, int T, int32_t* seq_start,
                               int32_t* seq_len, int32_t* chunk_off) {
    if (blockIdx.x != 0 || threadIdx.x != 0) return;
    int b = min(max(cu[0], 0), T);
    int acc = 0;
    chunk_off[0] = 0;
    for (int s = 0; s < n_seq; ++s) {
        int e = min(max(cu[s + 1], b), T);
        seq_start[s] = b;
        seq_len[s] = e - b;
        acc += (e - b + CH - 1) / CH;
        chunk_off[s + 1] = acc;
        b = e;
    }
}

// Stage rows [t0, t0+n) of a [*, H, D] io tensor (head h) into an LDS tile
// [64][LD]; rows n..63 are zero.
template <typename IO, int D, int LD>
__device__ __forceinline__ void stage_rows(IO (*dst)[LD], const IO* src, long t0, int n, int H, int h) {
    constexpr int VE = 16 / sizeof(IO);
    constexpr int VPR = D / VE;
    for (int i = threadIdx.x; i < CH * VPR; i += NT) {
        const int r = i / VPR, cv = i % VPR;
        uint4 val = make_uint4(0, 0, 0, 0);
        if (r < n) val = *reinterpret_cast<const uint4*>(src + ((t0 + r) * H + h) * (long)D + cv * VE);
        *reinterpret_cast<uint4*>(&dst[r][cv * VE]) = val;
    }
}

// ------------------------------------------------------------------ chunk terms
// One workgroup per (chunk slot, head): G, T = (I+A)^{-1} and P for one chunk.
template <typename IO, int DK>
__global__ __launch_bounds__(NT) void k_chunk_terms(Params p) {
    using M = Mma<IO>;
    constexpr int PAD = 16 / sizeof(IO);
    const int H = p.H;
    const int slot_x = blockIdx.x;
    const int gc = slot_x / H, h = slot_x % H;

    int s;
    if (p.ragged) {
        if (gc >= p.chunk_off[p.n_seq]) return;
        int lo = 0, hi = p.n_seq;
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (p.chunk_off[mid] <= gc) lo = mid; else hi = mid;
        }
        s = lo;
    } else {
        s = gc / p.NC;
    }
    long start;
    int len, cbase;
    seq_info(p, s, start, len, cbase);
    const int c = gc - cbase;
    const long t0 = start + (long)c * CH;
    const int n = min(CH, len - c * CH);

    __shared__ __attribute__((aligned(16))) IO sK[CH][DK + PAD];
    __shared__ __attribute__((aligned(16))) IO sQ[CH][DK + PAD];
    __shared__ __attribute__((aligned(16))) float sA[CH][CH + 4];
    __shared__ __attribute__((aligned(16))) float sTi[CH][CH + 4];
    __shared__ float sZ[4][16][17];
    __shared__ double sG[CH];
    __shared__ float sB[CH];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, lg = lane >> 4;
    const long slot = (long)gc * H + h;
    IO* Tg = reinterpret_cast<IO*>(p.wsT) + slot * CH * CH;
    IO* Pg = reinterpret_cast<IO*>(p.wsP) + slot * CH * CH;

    if (wave == 0) {
        float gv = 0.f, bv = 0.f;   // padded rows: no decay, no write
        if (lane < n) {
            gv = p.g[(t0 + lane) * H + h];
            bv = p.beta[(t0 + lane) * H + h];
        }
        double x = gv;   // inclusive prefix sum over the chunk, fp64
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const double y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        const double xn = __shfl(x, 63, 64);   // G_n (padded rows add nothing)
        sG[lane] = x;
        sB[lane] = bv;
        p.wsG[slot * 2 * CH + lane] = expf((float)x);
        p.wsG[slot * 2 * CH + CH + lane] = expf((float)(xn - x));
    }
    stage_rows<IO, DK, DK + PAD>(sK, reinterpret_cast<const IO*>(p.k), t0, n, H, h);
    stage_rows<IO, DK, DK + PAD>(sQ, reinterpret_cast<const IO*>(p.q), t0, n, H, h);
    // strictly-upper 16x16 blocks of P are zero
    for (int i = tid; i < CH * CH; i += NT) {
        const int r = i / CH, cc = i % CH;
        if ((cc >> 4) > (r >> 4)) Pg[i] = from_f<IO>(0.f);
    }
    __syncthreads();

    // 10 lower 16x16 blocks of K K^T (-> A) and of Q K^T (-> P)
    for (int job = wave; job < 20; job += 4) {
        const int which = job / 10;
        int t = job % 10, bi = 0;
        while (t > bi) { t -= bi + 1; ++bi; }
        const int bj = t;
        const IO(*X)[DK + PAD] = which ? sQ : sK;
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < DK / M::KS; ++kk) {
            const auto a = M::load(&X[bi * 16 + l16][kk * M::KS + lg * M::KL]);
            const auto b = M::load(&sK[bj * 16 + l16][kk * M::KS + lg * M::KL]);
            acc = M::mma(a, b, acc);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int r = bi * 16 + 4 * lg + e, i = bj * 16 + l16;
            if (which == 0) {
                sA[r][i] = (r > i) ? sB[r] * expf((float)(sG[r] - sG[i])) * acc[e] : 0.f;
            } else {
                Pg[r * CH + i] = from_f<IO>((r >= i) ? expf((float)(sG[r] - sG[i])) * acc[e] : 0.f);
            }
        }
    }
    __syncthreads();

    // T = (I + A)^{-1}, blocked by 16: the four diagonal blocks are inverted by
    // forward substitution (wave b, lane = column), then block row b follows from
    // T_bj = -T_bb * sum_{j <= m < b} A_bm T_mj with fp32 MFMA products.
    {
        const int b = wave;
        float x[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float acc = (r == l16) ? 1.f : 0.f;
#pragma unroll
            for (int i = 0; i < r; ++i) acc -= sA[16 * b + r][16 * b + i] * x[i];
            x[r] = acc;
        }
        if (lg == 0) {
#pragma unroll
            for (int r = 0; r < 16; ++r) sTi[16 * b + r][16 * b + l16] = x[r];
        }
    }
    __syncthreads();
    for (int b = 1; b < 4; ++b) {
        if (wave < b) {
            const int j = wave;
            floatx4 z = {0.f, 0.f, 0.f, 0.f};
            for (int m = j; m < b; ++m) {
#pragma unroll
                for (int kk = 0; kk < 4; ++kk)
                    z = __builtin_amdgcn_mfma_f32_16x16x4f32(sA[16 * b + l16][16 * m + 4 * kk + lg],
                                                             sTi[16 * m + 4 * kk + lg][16 * j + l16], z, 0, 0, 0);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) sZ[wave][4 * lg + e][l16] = z[e];
            __builtin_amdgcn_wave_barrier();   // LDS ops of one wave complete in order
            floatx4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
                t = __builtin_amdgcn_mfma_f32_16x16x4f32(sTi[16 * b + l16][16 * b + 4 * kk + lg],
                                                         sZ[wave][4 * kk + lg][l16], t, 0, 0, 0);
#pragma unroll
            for (int e = 0; e < 4; ++e) sTi[16 * b + 4 * lg + e][16 * j + l16] = -t[e];
        }
        __syncthreads();
    }
    for (int i = tid; i < CH * CH; i += NT) {
        const int r = i / CH, cc = i % CH;
        Tg[i] = from_f<IO>((cc >> 4) > (r >> 4) ? 0.f : sTi[r][cc]);
    }
}

// ------------------------------------------------------------------ state chain
// One workgroup per (sequence, head, 16-row slice of S); chunks in order.
template <typename IO, int DK>
__global__ __launch_bounds__(NT) void k_state_chain(Params p) {
    using M = Mma<IO>;
    constexpr int PAD = 16 / sizeof(IO);
    constexpr int NMT = DK / 16;          // 16-row tiles of S^T
    const int H = p.H, DV = p.DV, nsl = DV / SL;
    const int js = blockIdx.x % nsl;
    const int h = (blockIdx.x / nsl) % H;
    const int s = blockIdx.x / (nsl * H);

    long start;
    int len, cbase;
    seq_info(p, s, start, len, cbase);
    const int nc = (len + CH - 1) / CH;

    __shared__ __attribute__((aligned(16))) float sS[SL][DK + 4];   // rows js*16.. of S
    __shared__ __attribute__((aligned(16))) IO sK[CH][DK + PAD];
    __shared__ __attribute__((aligned(16))) IO sQ[CH][DK + PAD];
    __shared__ __attribute__((aligned(16))) IO sT[CH][CH + PAD];
    __shared__ __attribute__((aligned(16))) IO sP[CH][CH + PAD];
    __shared__ float sV[CH][SL + 1], sR[CH][SL + 1], sU[CH][SL + 1];
    __shared__ float sGam[CH], sDec[CH], sBeta[CH];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, lg = lane >> 4;
    const long srow0 = ((long)(s * H + h) * DV + js * SL) * DK;

    for (int i = tid; i < SL * DK; i += NT)
        sS[i / DK][i % DK] = p.S0 ? p.S0[srow0 + i] : 0.f;

    const IO* gv = reinterpret_cast<const IO*>(p.v);
    IO* go = reinterpret_cast<IO*>(p.o);

    for (int c = 0; c < nc; ++c) {
        const long t0 = start + (long)c * CH;
        const int n = min(CH, len - c * CH);
        const long slot = (long)(cbase + c) * H + h;
        __syncthreads();   // previous chunk done with every tile
        stage_rows<IO, DK, DK + PAD>(sK, reinterpret_cast<const IO*>(p.k), t0, n, H, h);
        stage_rows<IO, DK, DK + PAD>(sQ, reinterpret_cast<const IO*>(p.q), t0, n, H, h);
        {
            constexpr int VE = 16 / sizeof(IO), VPR = CH / VE;
            const IO* Tg = reinterpret_cast<const IO*>(p.wsT) + slot * CH * CH;
            const IO* Pg = reinterpret_cast<const IO*>(p.wsP) + slot * CH * CH;
            for (int i = tid; i < CH * VPR; i += NT) {
                const int r = i / VPR, cv = i % VPR;
                *reinterpret_cast<uint4*>(&sT[r][cv * VE]) = *reinterpret_cast<const uint4*>(Tg + r * CH + cv * VE);
                *reinterpret_cast<uint4*>(&sP[r][cv * VE]) = *reinterpret_cast<const uint4*>(Pg + r * CH + cv * VE);
            }
        }
        for (int i = tid; i < CH * SL; i += NT) {
            const int r = i / SL, j = i % SL;
            sV[r][j] = (r < n) ? to_f(gv[((t0 + r) * H + h) * (long)DV + js * SL + j]) : 0.f;
        }
        if (tid < CH) {
            sGam[tid] = p.wsG[slot * 2 * CH + tid];
            sDec[tid] = p.wsG[slot * 2 * CH + CH + tid];
            sBeta[tid] = (tid < n) ? p.beta[(t0 + tid) * H + h] : 0.f;
        }
        __syncthreads();

        // X = K S^T (tokens of tile `wave` x 16 value channels)
        floatx4 x = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < DK / M::KS; ++kk) {
            float sb[M::KL];
#pragma unroll
            for (int e = 0; e < M::KL; ++e) sb[e] = sS[l16][kk * M::KS + lg * M::KL + e];
            x = M::mma(M::load(&sK[wave * 16 + l16][kk * M::KS + lg * M::KL]), M::pack(sb), x);
        }
        // R = diag(beta) (V - diag(gamma) X)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int r = wave * 16 + 4 * lg + e;
            sR[r][l16] = sBeta[r] * (sV[r][l16] - sGam[r] * x[e]);
        }
        __syncthreads();

        // U = T R
        floatx4 u = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < CH / M::KS; ++kk) {
            float rb[M::KL];
#pragma unroll
            for (int e = 0; e < M::KL; ++e) rb[e] = sR[kk * M::KS + lg * M::KL + e][l16];
            u = M::mma(M::load(&sT[wave * 16 + l16][kk * M::KS + lg * M::KL]), M::pack(rb), u);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) sU[wave * 16 + 4 * lg + e][l16] = u[e];
        __syncthreads();

        // O = scale (diag(gamma) Q S^T + P U)
        floatx4 oq = {0.f, 0.f, 0.f, 0.f}, op = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < DK / M::KS; ++kk) {
            float sb[M::KL];
#pragma unroll
            for (int e = 0; e < M::KL; ++e) sb[e] = sS[l16][kk * M::KS + lg * M::KL + e];
            oq = M::mma(M::load(&sQ[wave * 16 + l16][kk * M::KS + lg * M::KL]), M::pack(sb), oq);
        }
#pragma unroll
        for (int kk = 0; kk < CH / M::KS; ++kk) {
            float ub[M::KL];
#pragma unroll
            for (int e = 0; e < M::KL; ++e) ub[e] = sU[kk * M::KS + lg * M::KL + e][l16];
            op = M::mma(M::load(&sP[wave * 16 + l16][kk * M::KS + lg * M::KL]), M::pack(ub), op);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int r = wave * 16 + 4 * lg + e;
            if (r < n)
                go[((t0 + r) * H + h) * (long)DV + js * SL + l16] =
                    from_f<IO>(p.scale * (sGam[r] * oq[e] + op[e]));
        }

        // S^T <- gamma_n S^T + K^T D U   (tiles of 16 key channels)
        const float gn = sGam[CH - 1];
        floatx4 acc[(NMT + 3) / 4];
#pragma unroll
        for (int m = 0; m < (NMT + 3) / 4; ++m) {
            const int mt = wave + 4 * m;
            acc[m] = floatx4{0.f, 0.f, 0.f, 0.f};
            if (mt < NMT) {
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[m][e] = gn * sS[l16][mt * 16 + 4 * lg + e];
#pragma unroll
                for (int kk = 0; kk < CH / M::KS; ++kk) {
                    float ka[M::KL], ub[M::KL];
#pragma unroll
                    for (int e = 0; e < M::KL; ++e) {
                        const int r = kk * M::KS + lg * M::KL + e;
                        ka[e] = to_f(sK[r][mt * 16 + l16]);
                        ub[e] = sDec[r] * sU[r][l16];
                    }
                    acc[m] = M::mma(M::pack(ka), M::pack(ub), acc[m]);
                }
            }
        }
        __syncthreads();   // every read of the old state is done
#pragma unroll
        for (int m = 0; m < (NMT + 3) / 4; ++m) {
            const int mt = wave + 4 * m;
            if (mt < NMT) {
#pragma unroll
                for (int e = 0; e < 4; ++e) sS[l16][mt * 16 + 4 * lg + e] = acc[m][e];
            }
        }
    }
    __syncthreads();
    if (p.ST)
        for (int i = tid; i < SL * DK; i += NT) p.ST[srow0 + i] = sS[i / DK][i % DK];
}

// ------------------------------------------------------------------ decode
// One token per sequence.  LPR lanes hold one state row as float4s; rows of S
// evolve independently: s_j <- alpha (s_j - beta (s_j.k) k) + beta v_j k.
template <typename IO, int DK>
__global__ __launch_bounds__(NT) void k_decode_step(const IO* __restrict__ q, const IO* __restrict__ k,
                                                    const IO* __restrict__ v, const float* __restrict__ g,
                                                    const float* __restrict__ beta, float* __restrict__ S,
                                                    IO* __restrict__ o, int DV, int rows_per_wg, float scale) {
    constexpr int LPR = DK / 4;        // lanes per row
    constexpr int RPP = NT / LPR;      // rows per pass of the workgroup
    const int bh = blockIdx.y;
    const int tid = threadIdx.x, sub = tid % LPR;
    float kv[4], qv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        kv[e] = to_f(k[(long)bh * DK + 4 * sub + e]);
        qv[e] = scale * to_f(q[(long)bh * DK + 4 * sub + e]);
    }
    const float a = expf(g[bh]);
    const float b = beta[bh];
    const int r0 = blockIdx.x * rows_per_wg;
    const int r1 = min(r0 + rows_per_wg, DV);
    for (int r = r0 + tid / LPR; r < r1; r += RPP) {
        float4* rowp = reinterpret_cast<float4*>(S + ((long)bh * DV + r) * DK) + sub;
        float4 sv = *rowp;
        float sk = sv.x * kv[0] + sv.y * kv[1] + sv.z * kv[2] + sv.w * kv[3];
#pragma unroll
        for (int m = LPR / 2; m >= 1; m >>= 1) sk += __shfl_xor(sk, m, 64);
        const float vj = to_f(v[(long)bh * DV + r]);
        const float cb = b * sk, wv = b * vj;
        sv.x = a * (sv.x - cb * kv[0]) + wv * kv[0];
        sv.y = a * (sv.y - cb * kv[1]) + wv * kv[1];
        sv.z = a * (sv.z - cb * kv[2]) + wv * kv[2];
        sv.w = a * (sv.w - cb * kv[3]) + wv * kv[3];
        *rowp = sv;
        float oj = sv.x * qv[0] + sv.y * qv[1] + sv.z * qv[2] + sv.w * qv[3];
#pragma unroll
        for (int m = LPR / 2; m >= 1; m >>= 1) oj += __shfl_xor(oj, m, 64);
        if (sub == 0) o[(long)bh * DV + r] = from_f<IO>(oj);
    }
}

// ------------------------------------------------------------------ host side
thread_local char g_err[512] = "";

gdn_status fail(gdn_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct Layout {
    long slots;          // chunk slots per head
    size_t meta, G, T, P, total;
};

// Workspace layout; returns false for arguments that are out of range.
bool ws_layout(int B, int T, int H, int dk, int dv, int n_seqs, int io, Layout* L) {
    (void)dk;
    (void)dv;
    const size_t esz = io == GDN_BF16 ? 2 : 4;
    const long cpt = ((long)T + CH - 1) / CH;
    L->slots = n_seqs > 0 ? cpt + n_seqs : (long)B * cpt;
    if (L->slots * (long)H > (1L << 24)) return false;
    const size_t per = (size_t)L->slots * H;
    L->meta = 0;
    L->G = n_seqs > 0 ? round_up((size_t)3 * (n_seqs + 1) * sizeof(int32_t), 256) : 0;
    L->T = L->G + round_up(per * 2 * CH * sizeof(float), 256);
    L->P = L->T + round_up(per * CH * CH * esz, 256);
    L->total = L->P + round_up(per * CH * CH * esz, 256);
    return true;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

template <typename IO, int DK>
void launch_prefill(const Params& p, long slots, hipStream_t st) {
    if (p.ragged)
        hipLaunchKernelGGL(k_ragged_setup, dim3(1), dim3(64), 0, st, p.cu, p.n_seq, p.T, p.seq_start,
                           p.seq_len, p.chunk_off);
    if (slots > 0 && p.T > 0)
        hipLaunchKernelGGL((k_chunk_terms<IO, DK>), dim3((unsigned)(slots * p.H)), dim3(NT), 0, st, p);
    hipLaunchKernelGGL((k_state_chain<IO, DK>), dim3((unsigned)(p.n_seq * p.H * (p.DV / SL))), dim3(NT), 0,
                       st, p);
}

template <typename IO, int DK>
void launch_decode(const void* q, const void* k, const void* v, const float* g, const float* beta,
                   float* S, void* o, int B, int H, int dv, float scale, hipStream_t st) {
    const int rows_per_wg = 32;
    dim3 grid((dv + rows_per_wg - 1) / rows_per_wg, B * H);
    hipLaunchKernelGGL((k_decode_step<IO, DK>), grid, dim3(NT), 0, st, (const IO*)q, (const IO*)k,
                       (const IO*)v, g, beta, S, (IO*)o, dv, rows_per_wg, scale);
}

}  // namespace

extern "C" int gdn_version(void) { return (0 << 16) | 1; }

extern "C" const char* gdn_status_string(int s) {
    switch (s) {
        case GDN_OK: return "GDN_OK";
        case GDN_ERR_INVALID_ARG: return "GDN_ERR_INVALID_ARG";
        case GDN_ERR_UNSUPPORTED: return "GDN_ERR_UNSUPPORTED";
        case GDN_ERR_WORKSPACE: return "GDN_ERR_WORKSPACE";
        case GDN_ERR_HIP: return "GDN_ERR_HIP";
        default: return "unknown status";
    }
}

extern "C" const char* gdn_last_error_message(void) { return g_err; }

static gdn_status check_dims(int dk, int dv) {
    if (dk < 1 || dv < 1) return fail(GDN_ERR_INVALID_ARG, "dk=%d dv=%d must be positive", dk, dv);
    if ((dk != 64 && dk != 128) || (dv != 64 && dv != 128))
        return fail(GDN_ERR_UNSUPPORTED, "dk=%d dv=%d: only 64 and 128 are implemented", dk, dv);
    return GDN_OK;
}

extern "C" size_t gdn_chunk_prefill_workspace_bytes(int B, int T, int H, int dk, int dv, int chunk,
                                                    int n_seqs, int io_dtype) {
    if (B < 1 || T < 0 || H < 1 || chunk != CH || n_seqs < 0 || (n_seqs > 0 && B != 1)) return 0;
    if (io_dtype != GDN_F32 && io_dtype != GDN_BF16) return 0;
    if ((dk != 64 && dk != 128) || (dv != 64 && dv != 128)) return 0;
    Layout L;
    if (!ws_layout(B, T, H, dk, dv, n_seqs, io_dtype, &L)) return 0;
    return L.total;
}

extern "C" gdn_status gdn_chunk_prefill(const void* q, const void* k, const void* v, const float* g,
                                        const float* beta, const float* S0, void* o, float* S_T, int B,
                                        int T, int H, int dk, int dv, int chunk, const int32_t* cu_seqlens,
                                        int n_seqs, int io_dtype, float scale, void* workspace,
                                        size_t workspace_bytes, void* stream) {
    g_err[0] = '\0';
    if (io_dtype != GDN_F32 && io_dtype != GDN_BF16)
        return fail(GDN_ERR_INVALID_ARG, "io_dtype=%d is neither GDN_F32 nor GDN_BF16", io_dtype);
    if (B < 1 || H < 1 || T < 0) return fail(GDN_ERR_INVALID_ARG, "B=%d H=%d T=%d out of range", B, H, T);
    gdn_status st = check_dims(dk, dv);
    if (st != GDN_OK) return st;
    if (chunk < 1) return fail(GDN_ERR_INVALID_ARG, "chunk=%d must be positive", chunk);
    if (chunk != CH) return fail(GDN_ERR_UNSUPPORTED, "chunk=%d: only 64 is implemented", chunk);
    if ((cu_seqlens == nullptr) != (n_seqs == 0))
        return fail(GDN_ERR_INVALID_ARG, "cu_seqlens and n_seqs=%d must be given together", n_seqs);
    if (n_seqs < 0) return fail(GDN_ERR_INVALID_ARG, "n_seqs=%d is negative", n_seqs);
    if (n_seqs > 0 && B != 1) return fail(GDN_ERR_INVALID_ARG, "ragged input needs B == 1 (got %d)", B);
    if (T > 0 && (!q || !k || !v || !g || !beta || !o))
        return fail(GDN_ERR_INVALID_ARG, "q, k, v, g, beta and o must be non-null");
    const void* vec_ptrs[] = {q, k, v, o, S0, S_T};   // read/written with 16-byte vectors
    for (const void* ptr : vec_ptrs)
        if (ptr && !aligned(ptr, 16)) return fail(GDN_ERR_INVALID_ARG, "tensor pointer %p is not 16-byte aligned", ptr);
    const void* scalar_ptrs[] = {g, beta, cu_seqlens};
    for (const void* ptr : scalar_ptrs)
        if (ptr && !aligned(ptr, 4)) return fail(GDN_ERR_INVALID_ARG, "pointer %p is not 4-byte aligned", ptr);
    const int n_seq = n_seqs > 0 ? n_seqs : B;
    if ((long)n_seq * H * (dv / SL) > (1L << 30)) return fail(GDN_ERR_UNSUPPORTED, "too many sequences x heads");
    if ((long)B * T * H > (1L << 40)) return fail(GDN_ERR_UNSUPPORTED, "B*T*H too large");
    Layout L;
    if (!ws_layout(B, T, H, dk, dv, n_seqs, io_dtype, &L))
        return fail(GDN_ERR_UNSUPPORTED, "too many chunks x heads for one call");
    if (workspace_bytes < L.total || (L.total > 0 && workspace == nullptr))
        return fail(GDN_ERR_WORKSPACE, "workspace of %zu bytes at %p; %zu bytes needed", workspace_bytes, workspace,
                    L.total);
    if (workspace && !aligned(workspace, 256)) return fail(GDN_ERR_INVALID_ARG, "workspace is not 256-byte aligned");

    Params p;
    p.q = q; p.k = k; p.v = v; p.g = g; p.beta = beta; p.S0 = S0; p.o = o; p.ST = S_T;
    p.B = B; p.T = T; p.H = H; p.DV = dv;
    p.n_seq = n_seq;
    p.ragged = n_seqs > 0;
    p.NC = (T + CH - 1) / CH;
    p.cu = cu_seqlens;
    char* ws = reinterpret_cast<char*>(workspace);
    p.seq_start = p.ragged ? reinterpret_cast<int32_t*>(ws) : nullptr;
    p.seq_len = p.ragged ? p.seq_start + (n_seqs + 1) : nullptr;
    p.chunk_off = p.ragged ? p.seq_len + (n_seqs + 1) : nullptr;
    p.wsG = reinterpret_cast<float*>(ws + L.G);
    p.wsT = ws + L.T;
    p.wsP = ws + L.P;
    p.scale = scale;
    if (L.total == 0) { p.wsG = nullptr; p.wsT = nullptr; p.wsP = nullptr; }

    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    if (io_dtype == GDN_BF16) {
        if (dk == 128) launch_prefill<bf16_t, 128>(p, L.slots, hs);
        else launch_prefill<bf16_t, 64>(p, L.slots, hs);
    } else {
        if (dk == 128) launch_prefill<float, 128>(p, L.slots, hs);
        else launch_prefill<float, 64>(p, L.slots, hs);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(GDN_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    return GDN_OK;
}

extern "C" gdn_status gdn_decode_step(const void* q, const void* k, const void* v, const float* g,
                                      const float* beta, float* S, void* o, int B, int H, int dk, int dv,
                                      int io_dtype, float scale, void* stream) {
    g_err[0] = '\0';
    if (io_dtype != GDN_F32 && io_dtype != GDN_BF16)
        return fail(GDN_ERR_INVALID_ARG, "io_dtype=%d is neither GDN_F32 nor GDN_BF16", io_dtype);
    if (B < 1 || H < 1) return fail(GDN_ERR_INVALID_ARG, "B=%d H=%d out of range", B, H);
    gdn_status st = check_dims(dk, dv);
    if (st != GDN_OK) return st;
    if (!q || !k || !v || !g || !beta || !S || !o)
        return fail(GDN_ERR_INVALID_ARG, "q, k, v, g, beta, S and o must be non-null");
    if (!aligned(S, 16)) return fail(GDN_ERR_INVALID_ARG, "state pointer %p is not 16-byte aligned", (const void*)S);
    const size_t esz = io_dtype == GDN_BF16 ? 2 : 4;
    const void* io_ptrs[] = {q, k, v, o};
    for (const void* ptr : io_ptrs)
        if (!aligned(ptr, esz)) return fail(GDN_ERR_INVALID_ARG, "pointer %p is not element-aligned", ptr);
    if (!aligned(g, 4) || !aligned(beta, 4)) return fail(GDN_ERR_INVALID_ARG, "g/beta are not 4-byte aligned");
    if ((long)B * H > 65535L * 1024) return fail(GDN_ERR_UNSUPPORTED, "B*H=%ld too large", (long)B * H);
    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    if (io_dtype == GDN_BF16) {
        if (dk == 128) launch_decode<bf16_t, 128>(q, k, v, g, beta, S, o, B, H, dv, scale, hs);
        else launch_decode<bf16_t, 64>(q, k, v, g, beta, S, o, B, H, dv, scale, hs);
    } else {
        if (dk == 128) launch_decode<float, 128>(q, k, v, g, beta, S, o, B, H, dv, scale, hs);
        else launch_decode<float, 64>(q, k, v, g, beta, S, o, B, H, dv, scale, hs);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(GDN_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    return GDN_OK;
}
