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
// When the chain alone would leave most compute units idle (few sequences and
// heads, many chunks), dense input takes the segment-parallel form: the
// sequence is cut into segments whose chains run at once, and the affine chunk
// map composes them (k_segment_prep, k_state_chain_pair*, k_segment_scan,
// k_segment_correct).
//
// Decode (k_decode_step) is the recurrence at T = 1: one pass over the state,
// row by row (rows of S never mix).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>
#include <time.h>

#include <atomic>
#include <type_traits>

#include "gdn.h"

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short short8 __attribute__((ext_vector_type(8)));
typedef uint16_t bf16_t;

constexpr int CH = 64;    // chunk length (tokens)
constexpr int NT = 256;   // threads per workgroup: 4 waves of 64
constexpr int SL = 16;    // state rows (value channels) per chain workgroup
constexpr int GS = 4 * CH;   // floats per (chunk slot, head) of the decay vectors: gamma, D, gamma s_k, gamma s_q

// Input transforms the kernels can apply themselves (bits of Params::pre, the
// flags of the _ex entry points): q and k scaled to unit length per (token,
// head), k / sqrt(|k|^2 + eps); and g, beta given as logits, g = -softplus(a),
// beta = sigmoid(b).
constexpr int PRE_L2 = 1, PRE_GATES = 2;
constexpr float L2_EPS = 1e-6f;
__device__ __forceinline__ float gate_g(float a) { return -(fmaxf(a, 0.f) + log1pf(expf(-fabsf(a)))); }
__device__ __forceinline__ float gate_beta(float b) { return 1.f / (1.f + expf(-b)); }

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
// Output layout of the 16x16 instructions (fp32 16x16x4, bf16 16x16x32): lane l
// holds D[4*(l/16) + e][l % 16], e = 0..3.  Lane l feeds row (A) / column (B)
// l % 16 and 1 (fp32) or 8 (bf16) contraction elements; which contraction
// indices a lane's elements stand for is a free choice as long as A and B agree.
__device__ __forceinline__ floatx4 f4(const void* ptr) { return *reinterpret_cast<const floatx4*>(ptr); }

// Fragment order of the lower-triangular 64x64 matrices W and P' for bf16 io.
// A 16x16x32 MFMA over a 64-long token contraction needs, for output row tile
// mt, contraction blocks kk = 0..mt/2 (the rest is zero): six fragments
// f = (mt, kk) = (0,0) (1,0) (2,0) (2,1) (3,0) (3,1).  Lane l, element e of
// fragment f holds M[16 mt + l%16][32 kk + 16 (e/4) + 4 (l/16) + e%4], so that
// contraction element e of lane group l/16 is token 32 kk + 16 (e/4) + 4 (l/16)
// + e%4 -- exactly the rows an MFMA accumulator tile pair holds in that lane.
constexpr int NFRAG = 6;
__host__ __device__ constexpr int frag_id(int mt, int kk) { return mt < 2 ? mt : 2 + 2 * (mt - 2) + kk; }
__device__ __forceinline__ int frag_mt(int f) { return f < 2 ? f : 2 + ((f - 2) >> 1); }
__device__ __forceinline__ int frag_kk(int f) { return f < 2 ? 0 : ((f - 2) & 1); }

// Elements per (chunk, head) slot of T and of P in the workspace.
template <typename IO> __host__ __device__ constexpr int tp_elems() { return sizeof(IO) == 2 ? NFRAG * 64 * 8 : CH * CH; }

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
    int st_t;          // S_T layout: 0 as declared; 1 transposed, [n, H, dk, DV] (key channel, then
                       // state row); 2 transposed in bf16 (the bf16 chain's identity run)
    int B, T, H, DV;
    int HK, G;         // key heads (q and k carry HK heads) and value heads per key head: head h reads key head h / G
    int n_seq;         // dense: B; ragged: number of packed sequences
    int ragged;
    int NC;            // dense: chunks per sequence
    int C;             // chunk length of the generic path (chunks other than 64)
    const int32_t* cu; // ragged: raw offsets (device)
    int32_t* seq_start;
    int32_t* seq_len;
    int32_t* chunk_off;  // [n_seq + 1], first chunk slot of each sequence
    int32_t* seq_perm;   // ragged: sequences by chunk count, longest first
    int32_t* cprefix;    // ragged: [cpt + 1] (sequence, chunk index < c) pair counts
    int cpt;             // chunks of the longest possible sequence
    float* wsG;          // [slot][H][GS]: gamma_r = exp(G_r), D_r = exp(G_n - G_r) (times s_k,r with PRE_L2
                         // in fp32 io), and with PRE_L2 gamma_r s_k,r and gamma_r s_q,r (s = 1 / |row|)
    void* wsT;           // [slot][H]: bf16 io W fragments; fp32 io T as high and low bf16 64 x 64 tiles
    void* wsP;           // [slot][H]: bf16 io P' fragments; fp32 io P as high and low bf16 64 x 64 tiles
    void* wsKQ;          // fp32 io: [slot][H][4][64][dk] bf16, K and Q as high and low parts (chain LDS order)
    uint64_t* flags;     // fused bf16 launch: [slot][H], = epoch once the slot's chunk terms are stored
    uint64_t epoch;      // per-call tag of those flags
    uint64_t* status;    // fused bf16 launch: the workspace's status word (= epoch when a wait gave up)
    int wait_bound;      // fused bf16 launch: most flag polls of one chain workgroup in the call
    int withhold;        // fused bf16 launch: chunk terms publish nothing (GDN_TEST_WITHHOLD)
    int npw;             // fused bf16 launch: chunk-terms workgroups ahead of the chain workgroups
    int xcd_items;       // fused bf16 launch: chunk-terms items assigned by XCD (dense, 8 | H, 8 | npw)
    float scale;
    int pre;             // PRE_L2 | PRE_GATES
    float* snaps;        // state snapshots [n_seq, n_snap, H, DV, dk] (the SNAP kernels only)
    int snap_every;      // ... after every snap_every chunks of a sequence, strictly inside it
    int n_snap;
};

// Entry i of a sequence table, read where every lane of the wave reads the same
// entry: held in a scalar register, so descriptors built from it stay scalar (a
// vector-register descriptor makes the compiler loop over its distinct values).
__device__ __forceinline__ int tab(const int32_t* a, long i) { return __builtin_amdgcn_readfirstlane(a[i]); }

// Sequence at rank r when sequences are taken longest first (ragged), else r.
__device__ __forceinline__ int seq_at_rank(const Params& p, int r) { return p.ragged ? tab(p.seq_perm, r) : r; }

// Work item k of the chunk terms in the order the chains consume them: chunk
// index within its sequence, then sequence rank, then head.
__device__ __forceinline__ long item_slot(const Params& p, long k) {
    const int H = p.H;
    int c, r;
    if (p.ragged) {
        int lo = 0, hi = p.cpt;   // largest c with cprefix[c] * H <= k
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if ((long)tab(p.cprefix, mid) * H <= k) lo = mid; else hi = mid;
        }
        c = lo;
        r = (int)((k - (long)tab(p.cprefix, c) * H) / H);
        return ((long)tab(p.chunk_off, tab(p.seq_perm, r)) + c) * H + (int)(k % H);
    }
    c = (int)(k / ((long)p.n_seq * H));
    r = (int)((k / H) % p.n_seq);
    return ((long)r * p.NC + c) * H + (int)(k % H);
}

__device__ __forceinline__ void seq_info(const Params& p, int s, long& start, int& len, int& cbase) {
    if (p.ragged) {
        start = tab(p.seq_start, s);
        len = tab(p.seq_len, s);
        cbase = tab(p.chunk_off, s);
    } else {
        start = (long)s * p.T;
        len = p.T;
        cbase = s * p.NC;
    }
}

// Sanitises the ragged offsets into a nondecreasing partition of [0, T] and
// lays out one workspace slot per chunk of every sequence.
// Exclusive scan of x[0..n) in place by one workgroup of NSET threads (each
// thread scans a contiguous segment; the segment totals by wave shuffles).
// reverse: the sum runs from the top index down.
constexpr int NSET = 1024;
__device__ void block_scan(int32_t* x, int n, bool reverse, int* part) {
    const int t = threadIdx.x, seg = (n + NSET - 1) / NSET;
    const int lo = t * seg, hi = min(n, lo + seg);
    auto at = [&](int i) -> int32_t& { return x[reverse ? n - 1 - i : i]; };
    int sum = 0;
    for (int i = lo; i < hi; ++i) sum += at(i);
    // exclusive scan of the segment totals: within each wave by shuffles, then over the wave totals
    const int lane = t & 63, wv = t >> 6;
    int inc = sum;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(inc, off, 64);
        if (lane >= off) inc += y;
    }
    if (lane == 63) part[wv] = inc;
    __syncthreads();
    if (t == 0) {
        int acc = 0;
        for (int i = 0; i < NSET / 64; ++i) {
            const int v = part[i];
            part[i] = acc;
            acc += v;
        }
    }
    __syncthreads();
    int acc = part[wv] + inc - sum;
    for (int i = lo; i < hi; ++i) {
        const int v = at(i);
        at(i) = acc;
        acc += v;
    }
    __syncthreads();
}

// Ragged sequence table: clamped starts and lengths, first chunk slot of each
// sequence; the sequences ordered by chunk count, longest first (perm); and
// prefix[c] = number of (sequence, chunk index c' < c) pairs, i.e. the sum over
// c' < c of the number of sequences with more than c' chunks.  ghist: cpt + 2
// ints of scratch, used when the histogram does not fit in LDS.  One workgroup
// of NSET threads.
__global__ __launch_bounds__(NSET) void k_ragged_setup(const int32_t* cu, int n_seq, int T, int32_t* seq_start,
                                                      int32_t* seq_len, int32_t* chunk_off, int32_t* perm,
                                                      int32_t* prefix, int32_t* ghist, int cpt, int ch) {
    __shared__ int part[NSET];
    __shared__ int scu[NSET + 1];
    __shared__ int shist[8192];
    int32_t* hist = cpt + 2 <= 8192 ? shist : ghist;   // the histogram in LDS when it fits
    const int t = threadIdx.x;
    // offsets clamped into a partition of [0, T]: a serial walk by thread 0 over
    // blocks of offsets that all threads fetch at once
    int b = 0, acc = 0;
    for (int s0 = 0; s0 < n_seq; s0 += NSET) {
        const int m = min(NSET, n_seq - s0);
        for (int i = t; i <= m; i += NSET) scu[i] = cu[s0 + i];
        __syncthreads();
        if (t == 0) {
            if (s0 == 0) {
                b = min(max(scu[0], 0), T);
                chunk_off[0] = 0;
            }
            for (int i = 0; i < m; ++i) {
                const int e = min(max(scu[i + 1], b), T);
                seq_start[s0 + i] = b;
                seq_len[s0 + i] = e - b;
                acc += (e - b + ch - 1) / ch;
                chunk_off[s0 + i + 1] = acc;
                b = e;
            }
        }
        __syncthreads();
    }
    for (int c = t; c <= cpt + 1; c += NSET) hist[c] = 0;
    __syncthreads();
    for (int s = t; s < n_seq; s += NSET) atomicAdd(&hist[(seq_len[s] + ch - 1) / ch], 1);   // counts <= cpt
    __syncthreads();
    // first rank of each chunk count, longest first: hist[n] <- #sequences with more than n chunks
    block_scan(hist, cpt + 1, true, part);
    for (int c = t; c <= cpt; c += NSET) prefix[c] = hist[c];
    __syncthreads();
    for (int s = t; s < n_seq; s += NSET) perm[atomicAdd(&hist[(seq_len[s] + ch - 1) / ch], 1)] = s;
    block_scan(prefix, cpt + 1, false, part);
}

// Stage rows [t0, t0+n) of two [*, H, D] io tensors (head h) into LDS tiles
// [64][LD]; rows n..63 are zero.  Every load is issued before the first LDS
// store, so the tiles cost one memory latency rather than one per pass.
template <typename IO, int D, int LD>
__device__ __forceinline__ void stage_rows2(IO (*dA)[LD], const IO* sA, IO (*dB)[LD], const IO* sB, long t0, int n,
                                            int H, int h) {
    constexpr int VE = 16 / sizeof(IO);
    constexpr int VPR = D / VE;
    constexpr int NPT = (CH * VPR + NT - 1) / NT;
    uint4 a[NPT], b[NPT];
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
        const int i = threadIdx.x + NT * j, r = i / VPR, cv = i % VPR;
        a[j] = b[j] = make_uint4(0, 0, 0, 0);
        if (i < CH * VPR && r < n) {
            const long off = ((t0 + r) * H + h) * (long)D + cv * VE;
            a[j] = *reinterpret_cast<const uint4*>(sA + off);
            b[j] = *reinterpret_cast<const uint4*>(sB + off);
        }
    }
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
        const int i = threadIdx.x + NT * j, r = i / VPR, cv = i % VPR;
        if (i < CH * VPR) {
            *reinterpret_cast<uint4*>(&dA[r][cv * VE]) = a[j];
            *reinterpret_cast<uint4*>(&dB[r][cv * VE]) = b[j];
        }
    }
}

// ------------------------------------------------------------------ bf16 operand helpers
typedef float floatx8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short short4v __attribute__((ext_vector_type(4)));
typedef int int4v __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
constexpr int NT_CHAIN = 512;
constexpr int RING = 4;
template <int N> struct Ic { static constexpr int value = N; };

__device__ __forceinline__ bf16x8 pack_bf16(floatx4 a, floatx4 b) {
    const floatx8 x = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_convertvector(x, bf16x8);
}
__device__ __forceinline__ bf16x8 join4(short4v a, short4v b) {
    const short8 x = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, x);
}
// whole-register select (a runtime index into a register array would be
// lowered element by element)
__device__ __forceinline__ bf16x8 sel(bool c, bf16x8 a, bf16x8 b) {
    return __builtin_bit_cast(bf16x8, c ? __builtin_bit_cast(int4v, a) : __builtin_bit_cast(int4v, b));
}
// Transpose read: within each 16-lane group, lane i element e receives element
// i%4 of the 8 bytes addressed by lane 4e + i/4 of the group.
__device__ __forceinline__ short4v lds_tr8(const bf16_t* ptr) {
    typedef __attribute__((address_space(3))) short4v lds_short4v;
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4v*)(ptr));
}
__device__ __forceinline__ float bf(short x) { return __uint_as_float((uint32_t)(uint16_t)x << 16); }
// Buffer resource over [base, base + bytes); loads past the end return zeros.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
}
// AUX: cache policy of the access (0: default; 17 = sc0 sc1: system coherent,
// bypassing the caches that other workgroups' data could be stale in)
template <int AUX = 0> __device__ __forceinline__ bf16x8 bload16(__amdgpu_buffer_rsrc_t r, int voff) {
    return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, AUX));
}
// global -> LDS without registers: lane l's 16 (4) bytes land at dst + 16 l (4 l)
template <int AUX = 0> __device__ __forceinline__ void bdma16(__amdgpu_buffer_rsrc_t r, void* dst, int voff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)dst, 16, voff, 0, 0, AUX);
}
template <int AUX = 0> __device__ __forceinline__ void bdma4(__amdgpu_buffer_rsrc_t r, void* dst, int voff) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)dst, 4, voff, 0, 0, AUX);
}
template <int AUX = 0> __device__ __forceinline__ void bstore16(bf16x8 v, __amdgpu_buffer_rsrc_t r, int voff) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(int4v, v), r, voff, 0, AUX);
}
template <int AUX = 0> __device__ __forceinline__ void bstore4(float v, __amdgpu_buffer_rsrc_t r, int voff) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, voff, 0, AUX);
}
// Workgroup barrier ordering LDS traffic only: the wave's own LDS operations
// complete, the compiler moves no memory access across it, and -- unlike
// __syncthreads() -- it does not wait for outstanding global loads or stores.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// x = hi + lo with hi = bf16(x), lo = bf16(x - hi): a product of two such pairs
// taken as hi*hi + hi*lo + lo*hi (the lo*lo term is below 2^-16 of it) gives fp32
// operands a relative error near 2^-16 from bf16 MFMA with fp32 accumulation
__device__ __forceinline__ void split8(floatx4 a, floatx4 b, bf16x8& hi, bf16x8& lo) {
    hi = pack_bf16(a, b);
    floatx4 ra, rb;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        ra[e] = a[e] - (float)hi[e];
        rb[e] = b[e] - (float)hi[4 + e];
    }
    lo = pack_bf16(ra, rb);
}
// The product of two split operands, its three terms into three accumulators (a sum
// over blocks is then three independent chains, not one): the product is a[0] + a[1] + a[2]
__device__ __forceinline__ void mma3x(bf16x8 ah, bf16x8 al, bf16x8 bh, bf16x8 bl, floatx4 (&a)[3]) {
    a[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, a[0], 0, 0, 0);
    a[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, a[1], 0, 0, 0);
    a[2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, a[2], 0, 0, 0);
}

// ------------------------------------------------------------------ fp32 io: operand images
// The fp32 chain takes K, Q, T and P as high and low bf16 parts, copied from the
// workspace straight into LDS; the chunk terms write them in the LDS order.
// K and Q (64 x dk): the 16-byte pieces of row r sit XOR-swizzled by f32_kq_swz(r),
// so the row reads (16 rows) and the transpose reads (4 rows, 4 pieces) of the chain
// meet no bank twice.  T and P (64 x 64): piece j of row r at j ^ (r % 8).
template <int DK> __device__ __forceinline__ int f32_kq_swz(int r) { return ((4 * (r & 3)) | ((r >> 2) & 3)) & (DK / 8 - 1); }
template <int DK> __device__ __forceinline__ int f32_kq_at(int r, int cc) {
    return r * DK + (((cc >> 3) ^ f32_kq_swz<DK>(r)) << 3) + (cc & 7);
}
__device__ __forceinline__ int f32_tp_at(int r, int cc) { return r * CH + (((cc >> 3) ^ (r & 7)) << 3) + (cc & 7); }

// ------------------------------------------------------------------ fp32 chunk terms
// One workgroup of eight waves per (chunk slot, head), fp32 io: G, T = (I+A)^{-1}
// and P for one chunk.
constexpr int NT_T32 = 512;
template <int DK>
__global__ __launch_bounds__(NT_T32) void k_chunk_terms(Params p) {
    using IO = float;
    const int H = p.H;
    const int slot_x = blockIdx.x;
    const int gc = slot_x / H, h = slot_x % H;

    int s;
    if (p.ragged) {
        if (gc >= tab(p.chunk_off, p.n_seq)) return;
        int lo = 0, hi = p.n_seq;
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (tab(p.chunk_off, mid) <= gc) lo = mid; else hi = mid;
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

    // K and Q are held as high and low bf16 parts (x = hi + lo, split8); once the
    // token-token products are in registers, A, T and P take the tiles' space (two
    // workgroups fit a CU's LDS).
    constexpr int KP = DK + 8;   // row pitch of the bf16 tiles
    constexpr int SZ_TILES = 4 * CH * KP * 2, SZ_MATS = 3 * CH * (CH + 4) * 4;
    __shared__ __attribute__((aligned(16))) char smem[SZ_TILES > SZ_MATS ? SZ_TILES : SZ_MATS];
    bf16_t(*sKh)[KP] = reinterpret_cast<bf16_t(*)[KP]>(smem);
    bf16_t(*sKl)[KP] = sKh + CH;
    bf16_t(*sQh)[KP] = sKh + 2 * CH;
    bf16_t(*sQl)[KP] = sKh + 3 * CH;
    float(*sA)[CH + 4] = reinterpret_cast<float(*)[CH + 4]>(smem);
    float(*sTi)[CH + 4] = sA + CH;
    float(*sP)[CH + 4] = sTi + CH;
    __shared__ float sZ[4][16][17];
    __shared__ double sG[CH];   // prefix sums of g in log2 units
    __shared__ float sB[CH], sD[CH], sSk[CH], sSq[CH];

    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, lg = lane >> 4;
    const long slot = (long)gc * H + h;
    bf16_t* Tg = reinterpret_cast<bf16_t*>(p.wsT) + slot * 2 * CH * CH;   // [hi | lo]
    bf16_t* Pg = reinterpret_cast<bf16_t*>(p.wsP) + slot * 2 * CH * CH;

    // K and Q rows: every load issued before the first store
    constexpr int NPR = DK / 8;                 // 8-channel pieces per row
    constexpr int NPC = CH * NPR / NT_T32;      // pieces per thread and tensor
    uint4 kv[NPC][2], qv[NPC][2];
    {
        const int HK = p.HK, hk = h / p.G;     // q and k carry HK heads; this head reads key head h / G
        const float* gk = reinterpret_cast<const float*>(p.k);
        const float* gq = reinterpret_cast<const float*>(p.q);
#pragma unroll
        for (int j = 0; j < NPC; ++j) {
            const int i = tid + NT_T32 * j, r = i / NPR, pc = i % NPR;
            kv[j][0] = kv[j][1] = qv[j][0] = qv[j][1] = make_uint4(0, 0, 0, 0);
            if (r < n) {   // rows past the chunk: zeros
                const long off = ((t0 + r) * HK + hk) * (long)DK + 8 * pc;
                kv[j][0] = *reinterpret_cast<const uint4*>(gk + off);
                kv[j][1] = *reinterpret_cast<const uint4*>(gk + off + 4);
                qv[j][0] = *reinterpret_cast<const uint4*>(gq + off);
                qv[j][1] = *reinterpret_cast<const uint4*>(gq + off + 4);
            }
        }
    }
    if (wave == 0) {
        float gv = 0.f, bv = 0.f;   // padded rows: no decay, no write
        if (lane < n) {
            gv = p.g[(t0 + lane) * H + h];
            bv = p.beta[(t0 + lane) * H + h];
            if (p.pre & PRE_GATES) {
                gv = gate_g(gv);
                bv = gate_beta(bv);
            }
        }
        double x = (double)gv * 1.4426950408889634;   // inclusive prefix sum over the chunk, fp64, log2 units
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const double y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        const double xn = __shfl(x, 63, 64);   // G_n (padded rows add nothing)
        sG[lane] = x;
        sB[lane] = bv;
        sD[lane] = __builtin_amdgcn_exp2f((float)(xn - x));
        p.wsG[slot * GS + lane] = __builtin_amdgcn_exp2f((float)x);
    }
    const bool l2 = p.pre & PRE_L2;
    {   // split each piece: the LDS tiles, and the chain's copy in its LDS order (f32_kq_at); with
        // PRE_L2 the squared row lengths, summed over the NPR consecutive lanes that hold a row
        bf16_t* kq = reinterpret_cast<bf16_t*>(p.wsKQ) + slot * 4 * CH * DK;   // [K hi | K lo | Q hi | Q lo]
#pragma unroll
        for (int j = 0; j < NPC; ++j) {
            const int i = tid + NT_T32 * j, r = i / NPR, pc = i % NPR;
            const int at = 8 * (r * NPR + (pc ^ f32_kq_swz<DK>(r)));
            const floatx4 k0 = __builtin_bit_cast(floatx4, kv[j][0]), k1 = __builtin_bit_cast(floatx4, kv[j][1]);
            const floatx4 q0 = __builtin_bit_cast(floatx4, qv[j][0]), q1 = __builtin_bit_cast(floatx4, qv[j][1]);
            bf16x8 hi, lo;
            split8(k0, k1, hi, lo);
            *reinterpret_cast<bf16x8*>(&sKh[r][8 * pc]) = hi;
            *reinterpret_cast<bf16x8*>(&sKl[r][8 * pc]) = lo;
            *reinterpret_cast<bf16x8*>(kq + at) = hi;
            *reinterpret_cast<bf16x8*>(kq + CH * DK + at) = lo;
            split8(q0, q1, hi, lo);
            *reinterpret_cast<bf16x8*>(&sQh[r][8 * pc]) = hi;
            *reinterpret_cast<bf16x8*>(&sQl[r][8 * pc]) = lo;
            *reinterpret_cast<bf16x8*>(kq + 2 * CH * DK + at) = hi;
            *reinterpret_cast<bf16x8*>(kq + 3 * CH * DK + at) = lo;
            if (l2) {
                const floatx4 kk2 = k0 * k0 + k1 * k1, qq2 = q0 * q0 + q1 * q1;
                float sk = kk2[0] + kk2[1] + kk2[2] + kk2[3], sq = qq2[0] + qq2[1] + qq2[2] + qq2[3];
#pragma unroll
                for (int m = 1; m < NPR; m <<= 1) {
                    sk += __shfl_xor(sk, m, 64);
                    sq += __shfl_xor(sq, m, 64);
                }
                if (pc == 0) {   // reciprocal row lengths; rows past the chunk: 0
                    sSk[r] = r < n ? 1.f / sqrtf(sk + L2_EPS) : 0.f;
                    sSq[r] = r < n ? 1.f / sqrtf(sq + L2_EPS) : 0.f;
                }
            }
        }
    }
    __syncthreads();
    if (tid < CH) {   // D (times s_k with PRE_L2), and the scaled decays the chain applies to K S^T and Q S^T
        const float gam = __builtin_amdgcn_exp2f((float)sG[tid]);
        p.wsG[slot * GS + CH + tid] = l2 ? sD[tid] * sSk[tid] : sD[tid];
        if (l2) {
            p.wsG[slot * GS + 2 * CH + tid] = gam * sSk[tid];
            p.wsG[slot * GS + 3 * CH + tid] = gam * sSq[tid];
        }
    }

    // 10 lower 16x16 blocks of K K^T (-> A) and of Q K^T (-> P): job = wave + 8 u < 20,
    // each as split bf16 products
    auto job_block = [](int job, int& which, int& bi, int& bj) {
        which = job / 10;
        int t = job % 10;
        bi = 0;
        while (t > bi) { t -= bi + 1; ++bi; }
        bj = t;
    };
    constexpr int NJ = 3;   // jobs per wave, at most
    floatx4 accs[NJ];
#pragma unroll
    for (int u = 0; u < NJ; ++u) {
        if (wave + 8 * u >= 20) break;
        int which, bi, bj;
        job_block(wave + 8 * u, which, bi, bj);
        const bf16_t(*Xh)[KP] = which ? sQh : sKh;
        const bf16_t(*Xl)[KP] = which ? sQl : sKl;
        const floatx4 z4 = {0.f, 0.f, 0.f, 0.f};
        floatx4 a3[3] = {z4, z4, z4};
#pragma unroll
        for (int kk = 0; kk < DK / 32; ++kk)
            mma3x(*reinterpret_cast<const bf16x8*>(&Xh[bi * 16 + l16][32 * kk + 8 * lg]),
                  *reinterpret_cast<const bf16x8*>(&Xl[bi * 16 + l16][32 * kk + 8 * lg]),
                  *reinterpret_cast<const bf16x8*>(&sKh[bj * 16 + l16][32 * kk + 8 * lg]),
                  *reinterpret_cast<const bf16x8*>(&sKl[bj * 16 + l16][32 * kk + 8 * lg]), a3);
        accs[u] = a3[0] + a3[1] + a3[2];
    }
    __syncthreads();   // every tile read done: A and P overwrite them
#pragma unroll
    for (int u = 0; u < NJ; ++u) {
        if (wave + 8 * u >= 20) break;
        int which, bi, bj;
        job_block(wave + 8 * u, which, bi, bj);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int r = bi * 16 + 4 * lg + e, i = bj * 16 + l16;
            const float nrm = l2 ? (which ? sSq[r] : sSk[r]) * sSk[i] : 1.f;
            if (which == 0) {
                sA[r][i] = (r > i) ? sB[r] * __builtin_amdgcn_exp2f((float)(sG[r] - sG[i])) * (nrm * accs[u][e]) : 0.f;
            } else {
                sP[r][i] = (r >= i) ? __builtin_amdgcn_exp2f((float)(sG[r] - sG[i])) * (nrm * accs[u][e]) : 0.f;
            }
        }
    }
    __syncthreads();

    // T = (I + A)^{-1}, blocked by 16: the four diagonal blocks are inverted by
    // forward substitution (wave b < 4, lane = column), then block row b follows from
    // T_bj = -T_bb * sum_{j <= m < b} A_bm T_mj with fp32 MFMA products.
    if (wave < 4) {
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
    // T and P for the chain: high and low bf16 parts in its LDS order (f32_tp_at), zero above the diagonal blocks
    for (int i = tid; i < CH * CH / 8; i += NT_T32) {
        const int r = i / (CH / 8), col = 8 * ((i % (CH / 8)) ^ (r & 7));
        const bool up = (col >> 4) > (r >> 4);
        const floatx4 z = {0.f, 0.f, 0.f, 0.f};
        bf16x8 hi, lo;
        split8(up ? z : f4(&sTi[r][col]), up ? z : f4(&sTi[r][col + 4]), hi, lo);
        *reinterpret_cast<bf16x8*>(Tg + 8 * i) = hi;
        *reinterpret_cast<bf16x8*>(Tg + CH * CH + 8 * i) = lo;
        split8(up ? z : f4(&sP[r][col]), up ? z : f4(&sP[r][col + 4]), hi, lo);
        *reinterpret_cast<bf16x8*>(Pg + 8 * i) = hi;
        *reinterpret_cast<bf16x8*>(Pg + CH * CH + 8 * i) = lo;
    }
}

// ------------------------------------------------------------------ fp32 state chain
// One workgroup of 8 waves per (sequence, head, 16-row slice of S); chunks in
// order (section 3.2): with S_c the state entering chunk c,
//   X = K S_c^T,  R = diag(beta) (V - diag(gamma_k) X),  U = T R,
//   S_{c+1}^T = gamma_n S_c^T + K^T diag(D) U,
//   O = scale (diag(gamma_q) Q S_c^T + P U).
// Waves 0-3 compute (wave w: token tile w of X, R, U and O, and the key tiles
// w + 4 m of the state update); waves 4-7 copy each chunk's operands into LDS
// with buffer loads to LDS: K, T and P as the high and low bf16 parts the chunk
// terms left in the workspace (in the LDS order), the V slice, the decay vectors
// and beta.  Each compute wave loads its own Q rows (split likewise) into
// registers at the start of the chunk.  Four barriers per chunk:
//   A_c  chunk c resident; the compute waves read every tile operand they need
//        (K rows and K^T fragments, T, P) into registers;
//   A'_c the copy waves issue chunk c+1's copy of K into the same tile;
//        the compute waves form X, R;
//   B_c  the copy waves issue the copies of T, P, V and the decay vectors (V and
//        the decay vectors alternate by chunk parity); the compute waves form U;
//   C_c  the compute waves update the state and form O.
// The copy waves wait for their copies before A_{c+1}.  The state slice stays in
// the compute waves' fp32 accumulators; S, R, U and D U go through LDS as high and
// low bf16 parts, split once by the wave that forms them.
// Every fp32 product is three bf16 MFMA products of high and low parts (mma3x);
// accumulation is fp32.
template <int DK> struct __attribute__((aligned(16))) F32ChainLds {
    bf16_t kq[2][CH * DK];                            // K hi, K lo (f32_kq_at)
    bf16_t tp[4][CH * CH];                            // T hi, T lo, P hi, P lo (f32_tp_at)
    bf16_t Sb[2][2][SL][DK + 8];                      // the slice of S, high and low parts, by chunk parity
    float V[2][CH * SL];                              // [token][value channel of the slice], by chunk parity
    float g[2][5 * CH];                               // gamma, D, gamma s_k, gamma s_q, beta; by chunk parity
    bf16_t Rb[2][SL][CH + 8];                         // R transposed, high and low parts
    bf16_t Ub[4][SL][CH + 8];                         // U and D U transposed, high and low parts
};

template <int DK, bool SNAP = false>
__device__ __forceinline__ void state_chain_f32(const Params& p, const int bid, F32ChainLds<DK>& lds) {
    constexpr int NKD = DK / 32;          // 32-long contraction blocks over the key channels
    constexpr int NMW = DK / 64;          // 16-key tiles of S^T per compute wave in the state update
    const int H = p.H, DV = p.DV, nsl = DV / SL;
    // slice-major: the slices of one (sequence, head) are congruent modulo H, so with
    // 8 | H they share an XCD (dispatch deals workgroups to the 8 XCDs in turn) and
    // its L2 copy of the head's operands
    const int s = bid / (nsl * H);
    const int js = (bid % (nsl * H)) / H;
    const int h = bid % H;
    long start;
    int len, cbase;
    seq_info(p, s, start, len, cbase);
    const int nc = (len + CH - 1) / CH;

    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, lg = lane >> 4;
    const long srow0 = ((long)(s * H + h) * DV + js * SL) * DK;

    if (wave >= 4) {
        // ------------------------------------------------ copy waves
        const int li = wave - 4;
        constexpr int KQB = 4 * CH * DK * 2, TPB = 2 * CH * CH * 2;   // bytes per (slot, head)
        // K (hi, lo): the first half of the K/Q image (the compute waves load their Q rows themselves)
        auto issue_k = [&](int c) {
            const long slot = (long)(cbase + c) * H + h;
            const auto rk = rsrc(reinterpret_cast<const char*>(p.wsKQ) + slot * KQB, KQB / 2);
#pragma unroll
            for (int i = li; i < KQB / 2048; i += 4) bdma16(rk, reinterpret_cast<char*>(&lds.kq[0][0]) + i * 1024, i * 1024 + lane * 16);
        };
        auto issue_rest = [&](int c) {
            const long slot = (long)(cbase + c) * H + h, t0 = start + (long)c * CH;
            const int n = min(CH, len - c * CH);
            const auto rt = rsrc(reinterpret_cast<const char*>(p.wsT) + slot * TPB, TPB);
            const auto rp = rsrc(reinterpret_cast<const char*>(p.wsP) + slot * TPB, TPB);
#pragma unroll
            for (int i = li; i < TPB / 1024; i += 4) {
                bdma16(rt, reinterpret_cast<char*>(&lds.tp[0][0]) + i * 1024, i * 1024 + lane * 16);
                bdma16(rp, reinterpret_cast<char*>(&lds.tp[2][0]) + i * 1024, i * 1024 + lane * 16);
            }
            // V rows 16 li .. 16 li + 15 of the slice (no value tensor: zeros); rows past the chunk read as zeros
            const long rb = (long)(n - 1) * H + 1;
            const auto rv = p.v ? rsrc(reinterpret_cast<const float*>(p.v) + (t0 * H + h) * DV, (uint32_t)(rb * DV * 4))
                                : rsrc(p.k, 0u);
            bdma16(rv, &lds.V[c & 1][16 * li * SL], ((16 * li + lane / 4) * H * DV + js * SL + 4 * (lane % 4)) * 4);
            if (li == 0) bdma16(rsrc(p.wsG + slot * GS, GS * 4), &lds.g[c & 1][0], lane * 16);
            if (li == 1) bdma4(rsrc(p.beta + t0 * H + h, (uint32_t)(rb * 4)), &lds.g[c & 1][4 * CH], lane * H * 4);
        };
        if (nc > 0) {
            issue_k(0);
            issue_rest(0);
        }
        // the copies of chunk c+1 go out over chunk c's phases (issuing them takes about as
        // long as their arithmetic; of the splits measured, K after A'_c and the rest after
        // B_c was the fastest)
        for (int c = 0; c < nc; ++c) {
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            lds_barrier();   // A_c
            lds_barrier();   // A'_c
            if (c + 1 < nc) issue_k(c + 1);
            lds_barrier();   // B_c
            if (c + 1 < nc) issue_rest(c + 1);
            lds_barrier();   // C_c
        }
        lds_barrier();   // F
        return;
    }

    // ------------------------------------------------ compute waves
    // S^T key tiles md = wave + 4 m stay in this wave's fp32 accumulators (element e of lane
    // group lg: key channel chan(md) + e, state row l16); each chunk publishes S as high and low
    // bf16 parts for every wave's B operands.
    auto chan = [&](int md) { return 32 * (md >> 1) + 8 * lg + 4 * (md & 1); };
    floatx4 acc[NMW];
#pragma unroll
    for (int m = 0; m < NMW; ++m)
        acc[m] = p.S0 ? *reinterpret_cast<const floatx4*>(p.S0 + srow0 + l16 * DK + chan(wave + 4 * m))
                      : floatx4{0.f, 0.f, 0.f, 0.f};
    auto put_split4 = [](bf16_t* hi, bf16_t* lo, floatx4 v) {   // 4 values -> 8 bytes of each part
        const bf16x4 h4 = __builtin_convertvector(v, bf16x4);
        floatx4 r;
#pragma unroll
        for (int e = 0; e < 4; ++e) r[e] = v[e] - (float)h4[e];
        *reinterpret_cast<bf16x4*>(hi) = h4;
        *reinterpret_cast<bf16x4*>(lo) = __builtin_convertvector(r, bf16x4);
    };
    auto publish_s = [&](int par) {
#pragma unroll
        for (int m = 0; m < NMW; ++m) put_split4(&lds.Sb[par][0][l16][chan(wave + 4 * m)], &lds.Sb[par][1][l16][chan(wave + 4 * m)], acc[m]);
    };
    if (nc > 0) publish_s(0);
    const bool l2 = p.pre & PRE_L2, gates = p.pre & PRE_GATES;
    const int row = wave * 16 + l16;   // token row of this lane's A operands
    const floatx4 z4 = {0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < nc; ++c) {
        const long t0 = start + (long)c * CH;
        const int n = min(CH, len - c * CH);
        const float* G = lds.g[c & 1];
        lds_barrier();   // A_c
        if constexpr (SNAP) {   // S_c, the state after c chunks
            if (c > 0 && c % p.snap_every == 0) {
                float* sn = p.snaps + (((long)s * p.n_snap + c / p.snap_every - 1) * H + h) * (long)DV * DK +
                            (long)(js * SL + l16) * DK;
#pragma unroll
                for (int m = 0; m < NMW; ++m) *reinterpret_cast<floatx4*>(sn + chan(wave + 4 * m)) = acc[m];
            }
        }
        // this wave's Q rows (high and low parts) straight from the workspace into registers, for
        // the output product at the end of the chunk (one LDS pass fewer)
        bf16x8 kh[NKD], kl[NKD], qh[NKD], ql[NKD], th[2], tl[2], ph[2], pl[2], kth[NMW][2], ktl[NMW][2];
        {
            constexpr int KQB = 4 * CH * DK * 2;
            const auto rq = rsrc(reinterpret_cast<const char*>(p.wsKQ) + ((long)(cbase + c) * H + h) * KQB + KQB / 2, KQB / 2);
#pragma unroll
            for (int kk = 0; kk < NKD; ++kk) {
                const int at = 2 * f32_kq_at<DK>(row, 32 * kk + 8 * lg);   // bytes
                qh[kk] = bload16(rq, at);
                ql[kk] = bload16(rq, CH * DK * 2 + at);
            }
        }
        // the tile operands into registers before A'_c (the copy waves refill the tiles after it)
#pragma unroll
        for (int kk = 0; kk < NKD; ++kk) {
            const int at = f32_kq_at<DK>(row, 32 * kk + 8 * lg);
            kh[kk] = *reinterpret_cast<const bf16x8*>(&lds.kq[0][at]);
            kl[kk] = *reinterpret_cast<const bf16x8*>(&lds.kq[1][at]);
        }
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const int at = f32_tp_at(row, 32 * kk + 8 * lg);
            th[kk] = *reinterpret_cast<const bf16x8*>(&lds.tp[0][at]);
            tl[kk] = *reinterpret_cast<const bf16x8*>(&lds.tp[1][at]);
            ph[kk] = *reinterpret_cast<const bf16x8*>(&lds.tp[2][at]);
            pl[kk] = *reinterpret_cast<const bf16x8*>(&lds.tp[3][at]);
        }
        // K^T fragments of key tiles md = wave + 4 m (transpose reads); contraction element j
        // of lane group lg in block kk is token 32 kk + 16 (j / 4) + 4 lg + j % 4
#pragma unroll
        for (int m = 0; m < NMW; ++m) {
            const int md = wave + 4 * m, col = 32 * (md >> 1) + 8 * (l16 & 3) + 4 * (md & 1);
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                const int o0 = f32_kq_at<DK>(32 * kk + 4 * lg + (l16 >> 2), col);
                const int o1 = f32_kq_at<DK>(32 * kk + 16 + 4 * lg + (l16 >> 2), col);
                kth[m][kk] = join4(lds_tr8(&lds.kq[0][o0]), lds_tr8(&lds.kq[0][o1]));
                ktl[m][kk] = join4(lds_tr8(&lds.kq[1][o0]), lds_tr8(&lds.kq[1][o1]));
            }
        }
        lds_barrier();   // A'_c
        // X = K S_c^T, S_c as B operands (key channel 32 kk + 8 lg + j, state row l16)
        bf16x8 sbh[NKD], sbl[NKD];
        floatx4 xa[3] = {z4, z4, z4};
#pragma unroll
        for (int kk = 0; kk < NKD; ++kk) {
            sbh[kk] = *reinterpret_cast<const bf16x8*>(&lds.Sb[c & 1][0][l16][32 * kk + 8 * lg]);
            sbl[kk] = *reinterpret_cast<const bf16x8*>(&lds.Sb[c & 1][1][l16][32 * kk + 8 * lg]);
            mma3x(kh[kk], kl[kk], sbh[kk], sbl[kk], xa);
        }
        {   // R = diag(beta) (V - diag(gamma_k) X) for tokens 16 wave + 4 lg + e; rows past the chunk: beta = 0
            const floatx4 x = xa[0] + xa[1] + xa[2];
            floatx4 rv;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r = wave * 16 + 4 * lg + e;
                const float braw = G[4 * CH + r];
                const float b = r < n ? (gates ? gate_beta(braw) : braw) : 0.f;
                rv[e] = b * (lds.V[c & 1][r * SL + l16] - (l2 ? G[2 * CH + r] : G[r]) * x[e]);
            }
            put_split4(&lds.Rb[0][l16][wave * 16 + 4 * lg], &lds.Rb[1][l16][wave * 16 + 4 * lg], rv);
        }
        lds_barrier();   // B_c

        // U = T R (k = token 32 kk + 8 lg + j); published as U and as D U
        {
            floatx4 ua[3] = {z4, z4, z4};
#pragma unroll
            for (int kk = 0; kk < 2; ++kk)
                mma3x(th[kk], tl[kk], *reinterpret_cast<const bf16x8*>(&lds.Rb[0][l16][32 * kk + 8 * lg]),
                      *reinterpret_cast<const bf16x8*>(&lds.Rb[1][l16][32 * kk + 8 * lg]), ua);
            const floatx4 u = ua[0] + ua[1] + ua[2];
            put_split4(&lds.Ub[0][l16][wave * 16 + 4 * lg], &lds.Ub[1][l16][wave * 16 + 4 * lg], u);
            put_split4(&lds.Ub[2][l16][wave * 16 + 4 * lg], &lds.Ub[3][l16][wave * 16 + 4 * lg],
                       f4(&G[CH + wave * 16 + 4 * lg]) * u);
        }
        lds_barrier();   // C_c

        // S^T <- gamma_n S^T + K^T (D U)
        {
            const float gn = G[CH - 1];
            bf16x8 dh[2], dl[2];
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                dh[kk] = join4(*reinterpret_cast<const short4v*>(&lds.Ub[2][l16][32 * kk + 4 * lg]),
                               *reinterpret_cast<const short4v*>(&lds.Ub[2][l16][32 * kk + 16 + 4 * lg]));
                dl[kk] = join4(*reinterpret_cast<const short4v*>(&lds.Ub[3][l16][32 * kk + 4 * lg]),
                               *reinterpret_cast<const short4v*>(&lds.Ub[3][l16][32 * kk + 16 + 4 * lg]));
            }
#pragma unroll
            for (int m = 0; m < NMW; ++m) {
                floatx4 sa[3] = {gn * acc[m], z4, z4};
#pragma unroll
                for (int kk = 0; kk < 2; ++kk) mma3x(kth[m][kk], ktl[m][kk], dh[kk], dl[kk], sa);
                acc[m] = sa[0] + sa[1] + sa[2];
            }
            publish_s((c + 1) & 1);
        }
        // O = scale (diag(gamma_q) Q S_c^T + P U)
        floatx4 qa[3] = {z4, z4, z4}, pa[3] = {z4, z4, z4};
#pragma unroll
        for (int kk = 0; kk < NKD; ++kk) mma3x(qh[kk], ql[kk], sbh[kk], sbl[kk], qa);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
            mma3x(ph[kk], pl[kk], *reinterpret_cast<const bf16x8*>(&lds.Ub[0][l16][32 * kk + 8 * lg]),
                  *reinterpret_cast<const bf16x8*>(&lds.Ub[1][l16][32 * kk + 8 * lg]), pa);
        {   // rows past the chunk fall outside the descriptor and are dropped
            const floatx4 oq = qa[0] + qa[1] + qa[2], op = pa[0] + pa[1] + pa[2];
            const auto ro = rsrc(reinterpret_cast<float*>(p.o) + (t0 * H + h) * DV, (uint32_t)((((long)n - 1) * H + 1) * DV * 4));
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r = wave * 16 + 4 * lg + e;
                const float ov = p.scale * ((l2 ? G[3 * CH + r] : G[r]) * oq[e] + op[e]);
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(ov), ro, (r * H * DV + js * SL + l16) * 4, 0, 0);
            }
        }
    }
    lds_barrier();   // F
    if (p.ST) {
#pragma unroll
        for (int m = 0; m < NMW; ++m) {
            if (p.st_t) {   // [n, H, dk, DV]
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    p.ST[srow0 - (long)js * SL * DK + (long)(chan(wave + 4 * m) + e) * DV + js * SL + l16] = acc[m][e];
            } else {
                *reinterpret_cast<floatx4*>(p.ST + srow0 + l16 * DK + chan(wave + 4 * m)) = acc[m];
            }
        }
    }
}

// One workgroup per CU (its LDS): two waves per SIMD.
template <int DK, bool SNAP = false>
__global__ __launch_bounds__(NT_CHAIN) __attribute__((amdgpu_waves_per_eu(1, 2))) void k_state_chain(Params p) {
    __shared__ F32ChainLds<DK> lds;
    state_chain_f32<DK, SNAP>(p, blockIdx.x, lds);
}

// ------------------------------------------------------------------ bf16 state chain
// One workgroup of 8 waves per (sequence, head, 16-row slice of S), bf16 io.
// Write S_c for the state entering chunk c, X_c = K_c S_c^T and
// R'_c = V_c - diag(gamma_c) X_c (section 3.2: V - diag(gamma) K S0^T).  Per chunk:
// D U = W_c R'_c (W_c = diag(D) T diag(beta)), S_{c+1}^T = gamma_n S_c^T + K_c^T D U,
// and X_{c+1} = K_{c+1} S_{c+1}^T for the next chunk's R'.
//  waves 0,1 ("chain"): wave w keeps the S^T rows of key-channel tiles
//    [NMD/2 w, NMD/2 (w+1)) as fp32 MFMA accumulators and the R' rows of token
//    tiles 2w, 2w+1.  After barrier A_c (R'_c complete) each forms D U from both
//    waves' R' tiles and updates its key tiles; it publishes its half of S_{c+1}
//    and forms its keys' share of X_{c+1} for all four token tiles.  At barrier
//    B_c the two waves swap the shares of each other's token tiles; each then
//    completes X_{c+1} and R'_{c+1} for its own tiles.  Every B operand (S, R',
//    D U) is packed from accumulators; the A operands are read in the matching
//    contraction order:
//      - token contractions: element e of lane group g in block kk is token
//        32 kk + 16 (e/4) + 4 g + e%4 (the rows an accumulator tile pair holds);
//      - key contractions: accumulator tile md, lane group g, element e holds
//        key channel 32 (md/2) + 8 g + 4 (md%2) + e, so a lane's 8 contraction
//        elements of block kk are the contiguous channels 32 kk + 8 g .. +7 and
//        the K (and Q) operands are single 16-byte reads.  K^T comes from the
//        row-major K tile through LDS transpose reads.
//  waves 2,3 ("output"): O_c^T = scale (S_c Q_c^T diag(gamma_c) + R'_c^T P'_c^T)
//    for one half of the chunk's tokens, from the published S_c and R'_c --
//    the operands swapped, so a lane ends up with 4 consecutive value channels
//    of one token and writes them with one 8-byte store.  Each stages its Q rows
//    in LDS two chunks ahead (buffer loads of whole cache lines: register loads
//    in the MFMA layout would read 64-byte halves) and loads its P' fragments
//    straight into registers, also two chunks ahead.
//  waves 4..7 ("loaders"): copy chunk c+3 (K, W, the V slice, gamma) into a
//    4-deep LDS ring with buffer loads to LDS, sharing the loads (one wave
//    alone issues global loads at about a third of a CU's rate).  In the one-
//    launch form wave 7 instead polls the chunk-terms flags a chunk ahead of
//    the three others' copies.
// Global loads use per-chunk buffer descriptors that end at row n-1 of the
// head, so the rows of a partial chunk read as zeros.  K rows sit in LDS with
// their 16-byte chunks XOR-swizzled by row, which keeps the transpose reads
// (4 rows, 4 chunks) free of bank conflicts.
// Two barriers per chunk.  At A_c, S_c and R'_c are complete (exchange buffers
// alternate by chunk parity) and every wave is done with chunk c-1, so the
// loaders refill that slot; chunk c+1, read during chunk c, was waited for
// before it.  B_c orders the chain waves' exchange of X_{c+1}; in the one-launch
// form the output waves issue their loads and stores after it, the loaders
// before it.  Barriers order LDS traffic only, so global loads and stores stay
// in flight across them.
// The chunk loop is unrolled by the ring depth so ring slots are constants.

// LDS of one chain workgroup
template <int DK> struct ChainLds {
    bf16_t sK[RING][CH * DK];     // ring of chunk inputs (slot = chunk % RING)
    bf16x8 sW[RING][NFRAG][64];   // diag(D) T diag(beta)
    bf16_t sV[RING][CH * SL];
    float sG[RING][CH];           // gamma_r
    float sGk[RING][CH];          // gamma_r s_k,r and gamma_r s_q,r (PRE_L2: K and Q taken unscaled)
    float sGq[RING][CH];
    bf16x8 sSf[2][DK / 32][64];   // S_c and R'_c as MFMA operands, by chunk parity
    bf16x8 sRf[2][2][64];
    floatx4 sY[2][2][64];         // each chain wave's share of X_{c+1} for the other wave's token tiles
    bf16_t sQ[2][2][32 * DK];     // Q rows of each output wave, by chunk parity
    int failed;                   // one launch: a wait for chunk terms gave up (set by the flag poller)
};

// Chain workgroup `bid`.  FUSED: the chunk terms come from workgroups of the
// same launch; a chunk's terms are read only once its flag carries this call's
// epoch, with loads that bypass the caches (their writers store the same way).
// IDENT: the identity run of the segment-parallel form -- values read as zeros
// and S_T stored transposed in bf16 (layout 2 of Params::st_t).  SNAP: the
// state is also stored after every snap_every chunks.  NORM (PRE_L2): K and Q
// rows arrive unscaled, so K S^T and Q S^T take the decays gamma s_k and gamma
// s_q (the chunk terms fold s_k into W).
template <int DK, bool FUSED, bool IDENT = false, bool SNAP = false, bool NORM = false>
__device__ __forceinline__ void state_chain_bf16(const Params& p, const int bid, ChainLds<DK>& lds) {
    constexpr int NKD = DK / 32;        // MFMA contraction blocks over the key channels
    constexpr int HKD = NKD / 2;        // ... whose S^T rows one chain wave keeps
    constexpr int HMD = DK / 32;        // 16-row S^T tiles per chain wave
    constexpr int NCH = DK / 8;         // 16-byte chunks per K row
    constexpr int RPI = 64 / NCH;       // rows per 1 KB direct load
    const int H = p.H, DV = p.DV;
    // Workgroups go longest sequence first (ragged), and within a sequence
    // slice-major, so the slices of one (sequence, head) are congruent modulo H:
    // with 8 | H they share an XCD (dispatch is round-robin over the 8 XCDs) and
    // its L2 copy of K, Q and the chunk matrices.
    const int per = H * (DV / SL);
    const int s = seq_at_rank(p, bid / per);
    const int js = (bid % per) / H;
    const int h = bid % H;
    long start;
    int len, cbase;
    seq_info(p, s, start, len, cbase);
    const int nc = (len + CH - 1) / CH;
    auto& sK = lds.sK;
    auto& sW = lds.sW;
    auto& sY = lds.sY;
    auto& sV = lds.sV;
    auto& sG = lds.sG;
    auto& sGk = NORM ? lds.sGk : lds.sG;   // decay of K S^T
    auto& sGq = NORM ? lds.sGq : lds.sG;   // decay of Q S^T
    auto& sSf = lds.sSf;
    auto& sRf = lds.sRf;
    auto& sQ = lds.sQ;
    constexpr int AUX = FUSED ? 17 : 0;   // sc0 sc1: coherent with the writers' stores

    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, lg = lane >> 4;
    const long srow0 = ((long)(s * H + h) * DV + js * SL) * DK;
    auto rows = [&](int c) { return min(CH, len - c * CH); };
    auto tok0 = [&](int c) { return start + (long)c * CH; };
    auto slot = [&](int c) { return (long)(cbase + c) * H + h; };
    auto swz = [](int r) { return ((4 * (r & 3)) | ((r >> 2) & 3)) & (NCH - 1); };
    // element offset of logical (row r, column cc) in a swizzled K tile
    auto kq = [&](int r, int cc) { return r * DK + (((cc >> 3) ^ swz(r)) << 3) + (cc & 7); };
    // descriptor over the rows of chunk c of this head in a [token][H][width] tensor
    auto crsrc = [&](const void* base, int width, int c) {
        return rsrc(reinterpret_cast<const bf16_t*>(base) + (tok0(c) * H + h) * width,
                    (uint32_t)(((long)(rows(c) - 1) * H + 1) * width * 2));
    };
    // ... and over the rows of q or k, which carry HK heads (this head reads key head h / G)
    const int HK = p.HK, hk = h / p.G;
    auto krsrc = [&](const void* base, int c) {
        return rsrc(reinterpret_cast<const bf16_t*>(base) + (tok0(c) * HK + hk) * DK,
                    (uint32_t)(((long)(rows(c) - 1) * HK + 1) * DK * 2));
    };
    // values; the identity run's read as zeros (a descriptor of no bytes)
    auto vrsrc = [&](int c) { return IDENT ? rsrc(p.k, 0u) : crsrc(p.v, DV, c); };

    if (FUSED && wave == 7) {
        // ------------------------------------------------ flag poller (one launch only)
        // Observes each chunk's flag one chunk before the loaders copy its terms
        // (the flag's memory round trip then overlaps a chunk's work, and the
        // loaders wait on their own copies only): chunks 0..2 before barrier P,
        // chunk 3 before the first chunk, chunk c+4 during chunk c.  The loaders'
        // copies of a chunk follow its observation through the barriers.
        // One bound on the polls of the whole call (each a memory round trip and a
        // short sleep: seconds in all at the default 2^22).  The chunk-terms
        // workgroups never wait and come first in the grid, so it is reached only
        // when they cannot run; then this workgroup reports instead of computing on
        // unpublished terms: the call's tag goes to the workspace's status word and
        // the output and chain waves, which read `failed` after the next barrier,
        // write NaN from there on.
        // The flag is a relaxed atomic: ordering comes from the cache-bypassing
        // (sc0 sc1) accesses on both sides -- the writer drains its bypassing stores
        // (vmcnt 0) before a barrier and the flag store, and the loaders read the terms
        // with bypassing loads after a barrier that follows this wave's observation
        // (lds_barrier is also a compiler memory barrier).  Acquire/release at agent
        // scope would add an L2 invalidate per poll and an L2 writeback per publication
        // on top of that; measured on the 10k 16-head call, 252 and 212 us against 141.
        int spins = p.wait_bound;
        if (lane == 0) lds.failed = 0;
        auto seen = [&](int c) {
            return __hip_atomic_load(&p.flags[slot(c)], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) == p.epoch;
        };
        auto wait_flag = [&](int c, bool ok) {
            while (!ok && spins > 0) {
                --spins;
                __builtin_amdgcn_s_sleep(2);
                ok = seen(c);
            }
            if (!ok && lane == 0) {
                lds.failed = 1;
                __hip_atomic_store(p.status, p.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
            }
        };
        if (FUSED && nc > 0)
            for (int c = 0; c < 3; ++c) wait_flag(min(c, nc - 1), seen(min(c, nc - 1)));
        lds_barrier();   // prologue P: chunks 0..2's terms published
        if (FUSED && nc > 0) wait_flag(min(3, nc - 1), seen(min(3, nc - 1)));
        lds_barrier();   // prologue 1
        lds_barrier();   // prologue 2
        for (int c = 0; c < nc; ++c) {
            lds_barrier();   // A_c
            const bool ok = FUSED ? seen(min(c + 4, nc - 1)) : true;
            lds_barrier();   // B_c
            if (FUSED) wait_flag(min(c + 4, nc - 1), ok);
        }
    } else if (wave >= 4) {
        // ------------------------------------------------ loaders
        // One wave issues global loads at about a third of a CU's rate, so NL
        // waves share the copies (four, or three beside the flag poller): K load
        // groups and W fragments with index = loader (mod NL), the two V loads on
        // loaders NL-2 and NL-1, gamma on loader 0.
        constexpr int NL = FUSED ? 3 : 4;
        const int li = wave - 4;
        const bf16_t* wsT = reinterpret_cast<const bf16_t*>(p.wsT);
        int koff[(NCH + NL - 1) / NL];   // loop-invariant byte offsets of this lane's K loads within a chunk
#pragma unroll
        for (int j = 0; j < (NCH + NL - 1) / NL; ++j) {
            const int r = RPI * (li + NL * j) + lane / NCH;
            koff[j] = (r * HK * DK + (((lane % NCH) ^ swz(r)) << 3)) * 2;
        }
        const int voff = ((32 * (li == NL - 1) + (lane >> 1)) * H * DV + js * SL + (lane & 1) * 8) * 2;
        // a chunk's copies of the inputs (K, V) and of its chunk terms (W, gamma)
        auto issue_in = [&](int c, auto SLOT, auto LI) {
            constexpr int sl = decltype(SLOT)::value, L = decltype(LI)::value;
            const auto rk = krsrc(p.k, c);
#pragma unroll
            for (int i = L; i < NCH; i += NL) bdma16(rk, &sK[sl][RPI * i * DK], koff[i / NL]);
            if constexpr (L >= NL - 2) bdma16(vrsrc(c), &sV[sl][32 * (L == NL - 1) * SL], voff);
        };
        auto issue_terms = [&](int c, auto SLOT, auto LI) {
            constexpr int sl = decltype(SLOT)::value, L = decltype(LI)::value;
            const long sc = slot(c);
            const auto rw = rsrc(wsT + sc * tp_elems<bf16_t>(), tp_elems<bf16_t>() * 2);
#pragma unroll
            for (int f = L; f < NFRAG; f += NL) bdma16<AUX>(rw, &sW[sl][f][0], (f * 64 + lane) * 16);
            const auto rg = rsrc(p.wsG + sc * GS, GS * 4);
            if constexpr (L == 0) bdma4<AUX>(rg, &sG[sl][0], lane * 4);
            if constexpr (NORM && L == 1) bdma4<AUX>(rg, &lds.sGk[sl][0], (2 * CH + lane) * 4);
            if constexpr (NORM && L == 2) bdma4<AUX>(rg, &lds.sGq[sl][0], (3 * CH + lane) * 4);
        };
        auto issue = [&](int c, auto SLOT, auto LI) {
            issue_in(c, SLOT, LI);
            issue_terms(c, SLOT, LI);
        };
        // After barrier A_c every wave is done with chunk c-1, whose slot is
        // (c+3) % RING: chunk c+3 is loaded there, and the wait leaves only
        // those loads in flight, so chunk c+2 has landed before barrier A_{c+1}.
        auto run = [&](auto LI) {
            constexpr int L = decltype(LI)::value;
            constexpr int NI = (NCH - L + NL - 1) / NL + (NFRAG - L + NL - 1) / NL + (L >= NL - 2) + (L == 0) +
                               (NORM && (L == 1 || L == 2));
            auto lstep = [&](int c, auto SLOT) {
                constexpr int bn = (decltype(SLOT)::value + 3) % RING;
                lds_barrier();   // A_c
                issue(min(c + 3, nc - 1), Ic<bn>{}, LI);
                lds_barrier();   // B_c
                asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NI) : "memory");
            };
            if (nc > 0) {   // the inputs need no chunk terms: copied while those are formed
                issue_in(0, Ic<0>{}, LI);
                issue_in(min(1, nc - 1), Ic<1>{}, LI);
                issue_in(min(2, nc - 1), Ic<2>{}, LI);
            }
            lds_barrier();   // prologue P
            if (nc > 0) {
                issue_terms(0, Ic<0>{}, LI);
                issue_terms(min(1, nc - 1), Ic<1>{}, LI);
                issue_terms(min(2, nc - 1), Ic<2>{}, LI);
            }
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            lds_barrier();   // prologue 1: chunks 0, 1 and 2 resident
            lds_barrier();   // prologue 2: S_0 halves visible
            for (int c = 0; c < nc; c += RING) {
                lstep(c, Ic<0>{});
                if (c + 1 < nc) lstep(c + 1, Ic<1>{});
                if (c + 2 < nc) lstep(c + 2, Ic<2>{});
                if (c + 3 < nc) lstep(c + 3, Ic<3>{});
            }
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        };
        switch (li) {
            case 0: run(Ic<0>{}); break;
            case 1: run(Ic<1>{}); break;
            case 2: run(Ic<2>{}); break;
            default:
                if constexpr (NL > 3) run(Ic<3>{});
                break;
        }
    } else if (wave < 2) {
        // ------------------------------------------------ chain waves
        // (one instance per wave, so the wave's half is a constant: no selects)
        auto chain = [&](auto WI) {
            constexpr int w = decltype(WI)::value;
            auto chan = [&](int md) { return 32 * (md >> 1) + 8 * lg + 4 * (md & 1); };   // + e
            floatx4 acc[HMD];
#pragma unroll
            for (int m = 0; m < HMD; ++m) {
                acc[m] = floatx4{0.f, 0.f, 0.f, 0.f};
                if (p.S0) acc[m] = *reinterpret_cast<const floatx4*>(p.S0 + srow0 + l16 * DK + chan(w * HMD + m));
            }
            // loop-invariant LDS offsets of this lane's operands
            int offT[HMD][2][2];      // K^T fragments of this wave's key tiles (transpose reads)
            int offV[2];              // V rows of this wave's token tiles (transpose reads)
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int mt = 2 * w + i;
                offV[i] = (16 * mt + 4 * lg + (l16 >> 2)) * SL + 4 * (l16 & 3);
            }
#pragma unroll
            for (int m = 0; m < HMD; ++m) {
                const int md = w * HMD + m;
#pragma unroll
                for (int kk = 0; kk < 2; ++kk)
#pragma unroll
                    for (int h2 = 0; h2 < 2; ++h2)
                        offT[m][kk][h2] = kq(32 * kk + 16 * h2 + 4 * lg + (l16 >> 2),
                                             32 * (md >> 1) + 8 * (l16 & 3) + 4 * (md & 1));
            }
            bf16x8 sfo[HKD], rfo;   // this wave's halves of S_c and R'_c
            auto publish_s = [&](int par) {
#pragma unroll
                for (int k2 = 0; k2 < HKD; ++k2) {
                    sfo[k2] = pack_bf16(acc[2 * k2], acc[2 * k2 + 1]);
                    sSf[par][w * HKD + k2][lane] = sfo[k2];
                }
            };
            // R' rows of this wave's token tiles from X = K S^T: V - diag(gamma) X
            struct VG {
                short4v vv[2];
                floatx4 gm[2];
            };
            auto load_vg = [&](int bn) {
                VG r;
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    r.vv[i] = lds_tr8(&sV[bn][offV[i]]);
                    r.gm[i] = *reinterpret_cast<const floatx4*>(&sGk[bn][16 * (2 * w + i) + 4 * lg]);
                }
                return r;
            };
            auto rprime = [&](const floatx4 (&y)[2], const VG& vg) {
                floatx4 rr[2];
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int e = 0; e < 4; ++e) rr[i][e] = bf(vg.vv[i][e]) - vg.gm[i][e] * y[i][e];
                return pack_bf16(rr[0], rr[1]);
            };
            lds_barrier();   // prologue P: chunks 0..2's terms published
            lds_barrier();   // prologue 1: chunks 0, 1 and 2 resident
            if (nc > 0) publish_s(0);
            lds_barrier();   // prologue 2: S_0 halves visible
            if (nc > 0) {    // R'_0 = V_0 - diag(gamma_0) K_0 S_0^T for this wave's token tiles
                bf16x8 sfx[HKD];
#pragma unroll
                for (int k2 = 0; k2 < HKD; ++k2) sfx[k2] = sSf[0][(1 - w) * HKD + k2][lane];
                floatx4 y[2];
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    y[i] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int k2 = 0; k2 < HKD; ++k2) {
                        const int r = 16 * (2 * w + i) + l16;
                        y[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            *reinterpret_cast<const bf16x8*>(&sK[0][kq(r, 32 * (w * HKD + k2) + 8 * lg)]), sfo[k2], y[i], 0, 0, 0);
                        y[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            *reinterpret_cast<const bf16x8*>(&sK[0][kq(r, 32 * ((1 - w) * HKD + k2) + 8 * lg)]), sfx[k2], y[i],
                            0, 0, 0);
                    }
                }
                rfo = rprime(y, load_vg(0));
                sRf[0][w][lane] = rfo;
            }
            // K_{c+1} rows of all four token tiles over this wave's key blocks (the
            // partial products X_{c+1} = K_{c+1} S_{c+1}^T the waves exchange)
            int offY[4][HKD];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                for (int k2 = 0; k2 < HKD; ++k2) offY[mt][k2] = kq(16 * mt + l16, 32 * (w * HKD + k2) + 8 * lg);
            auto cstep = [&](int c, auto SLOT) {   // chunk c = SLOT (mod RING)
                constexpr int b = decltype(SLOT)::value, bn = (b + 1) % RING, x2 = b & 1;
                lds_barrier();   // barrier A_c: S_c halves and R'_c visible
                const bf16x8 rfx = sRf[x2][1 - w][lane];
                const bf16x8 rf0 = sel(w == 0, rfo, rfx), rf1 = sel(w == 0, rfx, rfo);
                const float gn = sG[b][CH - 1];
                bf16x8 wf[NFRAG], ka[HMD][2], ky[4][HKD];
#pragma unroll
                for (int f = 0; f < NFRAG; ++f) wf[f] = sW[b][f][lane];
#pragma unroll
                for (int m = 0; m < HMD; ++m)
#pragma unroll
                    for (int kk = 0; kk < 2; ++kk)
                        ka[m][kk] = join4(lds_tr8(&sK[b][offT[m][kk][0]]), lds_tr8(&sK[b][offT[m][kk][1]]));
                // chunk c+1's operands are resident since barrier A_c: read them ahead of
                // the products that need them
#pragma unroll
                for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                    for (int k2 = 0; k2 < HKD; ++k2) ky[mt][k2] = *reinterpret_cast<const bf16x8*>(&sK[bn][offY[mt][k2]]);
                const VG vg = load_vg(bn);
                // D U = W R' (lower triangular: tile mt needs blocks 0..mt/2); S^T <- gn S^T + K^T (D U)
                floatx4 du[4];
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    du[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[frag_id(mt, 0)], rf0, floatx4{0.f, 0.f, 0.f, 0.f},
                                                                     0, 0, 0);
                    if (mt >= 2) du[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[frag_id(mt, 1)], rf1, du[mt], 0, 0, 0);
                }
                const bf16x8 df0 = pack_bf16(du[0], du[1]), df1 = pack_bf16(du[2], du[3]);
#pragma unroll
                for (int m = 0; m < HMD; ++m) {
                    acc[m] *= gn;
                    acc[m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[m][0], df0, acc[m], 0, 0, 0);
                    acc[m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[m][1], df1, acc[m], 0, 0, 0);
                }
                if constexpr (SNAP) {   // S_{c+1}, the state after c + 1 chunks
                    if ((c + 1) % p.snap_every == 0 && c + 1 < nc) {
                        float* sn = p.snaps + (((long)s * p.n_snap + (c + 1) / p.snap_every - 1) * H + h) * (long)DV * DK +
                                    (long)(js * SL + l16) * DK;
#pragma unroll
                        for (int m = 0; m < HMD; ++m) *reinterpret_cast<floatx4*>(sn + chan(w * HMD + m)) = acc[m];
                    }
                }
                // S_{c+1}: this wave's half for the output waves, and its share of X_{c+1}
                publish_s(1 - x2);
                floatx4 yp[4];
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    yp[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int k2 = 0; k2 < HKD; ++k2)
                        yp[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ky[mt][k2], sfo[k2], yp[mt], 0, 0, 0);
                }
                // (whole-value selects: a runtime index into a register array would go to scratch)
                floatx4 own[2], oth[2];
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    own[i] = w == 0 ? yp[i] : yp[2 + i];
                    oth[i] = w == 0 ? yp[2 + i] : yp[i];
                    sY[w][i][lane] = oth[i];   // the other wave's token tiles
                }
                lds_barrier();   // barrier B_c: both waves' shares of X_{c+1} visible
                floatx4 y[2];
#pragma unroll
                for (int i = 0; i < 2; ++i) y[i] = own[i] + sY[1 - w][i][lane];
                // R'_{c+1}, published for chunk c+1
                rfo = rprime(y, vg);
                sRf[1 - x2][w][lane] = rfo;
            };
            for (int c = 0; c < nc; c += RING) {
                cstep(c, Ic<0>{});
                if (c + 1 < nc) cstep(c + 1, Ic<1>{});
                if (c + 2 < nc) cstep(c + 2, Ic<2>{});
                if (c + 3 < nc) cstep(c + 3, Ic<3>{});
            }
            if constexpr (IDENT) {
                bf16_t* st = reinterpret_cast<bf16_t*>(p.ST) + srow0 - (long)js * SL * DK + js * SL + l16;
#pragma unroll
                for (int m = 0; m < HMD; ++m)
#pragma unroll
                    for (int e = 0; e < 4; ++e) st[(long)(chan(w * HMD + m) + e) * DV] = from_f<bf16_t>(acc[m][e]);
            } else if (p.ST) {
                if (FUSED && lds.failed)
#pragma unroll
                    for (int m = 0; m < HMD; ++m) acc[m] = floatx4{__builtin_nanf(""), __builtin_nanf(""), __builtin_nanf(""), __builtin_nanf("")};
#pragma unroll
                for (int m = 0; m < HMD; ++m)
                    *reinterpret_cast<floatx4*>(p.ST + srow0 + l16 * DK + chan(w * HMD + m)) = acc[m];
            }
        };
        if (wave == 0) chain(Ic<0>{});
        else chain(Ic<1>{});
    } else {
        // ------------------------------------------------ output waves
        // Wave 2 + o handles token tiles 2o, 2o + 1 (rows 32o .. 32o + 31).  Its Q
        // rows are staged in LDS by buffer loads (whole 128-byte lines, XOR-swizzled
        // like K), two chunks ahead in two buffers.  P' token tile mt needs fragments
        // (mt, 0..mt/2): wave 2 fragments 0, 1; wave 3 fragments 2, 3, 4, 5.
        auto run = [&](auto OW) {
            constexpr int ow = decltype(OW)::value, NPP = ow ? 4 : 2;
            const bf16_t* wsP = reinterpret_cast<const bf16_t*>(p.wsP);

            int qoff[32 / RPI];   // byte offsets of this lane's Q row loads within a chunk
#pragma unroll
            for (int j = 0; j < 32 / RPI; ++j) {
                const int r = RPI * j + lane / NCH;
                qoff[j] = ((32 * ow + r) * HK * DK + (((lane % NCH) ^ swz(r)) << 3)) * 2;
            }
            auto load_q = [&](int c, bf16_t* sq) {
                const auto rq = krsrc(p.q, c);
#pragma unroll
                for (int j = 0; j < 32 / RPI; ++j) bdma16(rq, sq + RPI * j * DK, qoff[j]);
            };
            auto load_p = [&](int c, bf16x8(&pa)[NPP]) {
                const auto rp = rsrc(wsP + slot(c) * tp_elems<bf16_t>(), tp_elems<bf16_t>() * 2);
#pragma unroll
                for (int k = 0; k < NPP; ++k) pa[k] = bload16<AUX>(rp, ((ow ? 2 + k : k) * 64 + lane) * 16);
            };
            // In chunk c this wave issues the P' loads of chunk c+2, into register
            // set (c+2) % 4, the Q copy of chunk c+2, into the buffer chunk c's rows
            // leave, and chunk c's output stores: in one launch all after barrier
            // B_c (the loader waves' copies go out between A_c and B_c), with two
            // launches the loads as soon as chunk c's rows are read and the stores
            // as the outputs are formed.  Loads complete in issue order, so at a chunk's start
            // waiting until NPP + NQ remain covers its P' loads and its Q copy.
            // (Chunk c+2's terms are published: in one launch the flag poller saw
            // its flag two chunks earlier; with two launches the chunk terms came
            // first.)
            constexpr int NQ = 32 / RPI;
            bf16x8 pS[RING][NPP];   // P' fragments by ring slot
            auto ostep = [&](int c, auto SLOT) {
                constexpr int b = decltype(SLOT)::value, x2 = b & 1;
                const bf16x8(&pa)[NPP] = pS[b];
                bf16_t* sq = sQ[x2][ow];
                lds_barrier();   // barrier A_c: S_c and R'_c visible
                asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NPP + NQ) : "memory");   // Q_c staged, P'_c loaded
                bf16x8 qa[2][NKD];
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int kk = 0; kk < NKD; ++kk)
                        qa[i][kk] = *reinterpret_cast<const bf16x8*>(sq + kq(16 * i + l16, 32 * kk + 8 * lg));
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // staging buffer read: free for Q_{c+2}
                if constexpr (!FUSED) {
                    load_p(min(c + 2, nc - 1), pS[(b + 2) % RING]);
                    load_q(min(c + 2, nc - 1), sq);
                }
                const bf16x8 rf0 = sRf[x2][0][lane], rf1 = sRf[x2][1][lane];
                const auto ro = crsrc(p.o, DV, c);
                typedef int int2v __attribute__((ext_vector_type(2)));
                int2v ovs[2];
                auto store_o = [&](int i) {   // 4 value channels of token 16 (2 ow + i) + l16
                    __builtin_amdgcn_raw_buffer_store_b64(ovs[i], ro, ((16 * (2 * ow + i) + l16) * H * DV + js * SL + 4 * lg) * 2,
                                                          0, 0);
                };
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int mt = 2 * ow + i, tok = 16 * mt + l16;
                    const float gm = sGq[b][tok];
                    floatx4 oq = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int kk = 0; kk < NKD; ++kk)
                        oq = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sSf[x2][kk][lane], qa[i][kk], oq, 0, 0, 0);
                    floatx4 op;
                    if constexpr (ow == 0) {
                        op = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rf0, pa[i], floatx4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                    } else {   // fragments (mt, 0) = pa[2 i], (mt, 1) = pa[2 i + 1]
                        op = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rf0, pa[2 * i], floatx4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                        op = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rf1, pa[2 * i + 1], op, 0, 0, 0);
                    }
                    floatx4 ov = p.scale * (gm * oq + op);   // value channels 4 lg .. 4 lg + 3 of token tok
                    if (FUSED && lds.failed) ov = floatx4{__builtin_nanf(""), __builtin_nanf(""), __builtin_nanf(""), __builtin_nanf("")};
                    ovs[i] = __builtin_bit_cast(int2v, __builtin_convertvector(ov, bf16x4));
                    if constexpr (!FUSED) store_o(i);
                }
                lds_barrier();   // B_c (the chain waves' exchange of X_{c+1}); S_c and R'_c are no longer read
                if constexpr (FUSED) {
                    load_p(min(c + 2, nc - 1), pS[(b + 2) % RING]);
                    load_q(min(c + 2, nc - 1), sq);
                    store_o(0);
                    store_o(1);
                }
            };
            if (nc > 0) {   // Q is an input: staged while the first chunk terms are formed
                load_q(0, sQ[0][ow]);
                load_q(min(1, nc - 1), sQ[1][ow]);
            }
            lds_barrier();   // prologue P: chunks 0..2's terms published
            lds_barrier();   // prologue 1
            if (nc > 0) {
                load_p(0, pS[0]);
                load_p(min(1, nc - 1), pS[1]);
            }
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // (the first chunks' waits assume the steady-state order)
            lds_barrier();   // prologue 2
            for (int c = 0; c < nc; c += RING) {   // unrolled so ring slot and fragment set are constants
                ostep(c, Ic<0>{});
                if (c + 1 < nc) ostep(c + 1, Ic<1>{});
                if (c + 2 < nc) ostep(c + 2, Ic<2>{});
                if (c + 3 < nc) ostep(c + 3, Ic<3>{});
            }
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        };
        if (wave == 2) run(Ic<0>{});
        else run(Ic<1>{});
    }
}

// One workgroup per CU (its LDS), so two waves per SIMD: the register budget is that of two waves.
template <int DK, bool SNAP = false, bool NORM = false>
__global__ __launch_bounds__(NT_CHAIN) __attribute__((amdgpu_waves_per_eu(1, 2))) void k_state_chain_bf16(Params p) {
    __shared__ ChainLds<DK> lds;
    state_chain_bf16<DK, false, false, SNAP, NORM>(p, blockIdx.x, lds);
}

// ------------------------------------------------------------------ bf16 chunk terms
// One workgroup (4 waves) per (chunk slot, head), bf16 io.  Produces for the
// state chain gamma_r and exp(G_n - G_r), and in MFMA fragment order
//     W  = diag(D) T diag(beta)     lower triangular, 6 fragments
//     P' = P T diag(beta)           lower triangular, 6 fragments
// with T = (I + A)^{-1}.
// Stages: K and Q arrive by buffer loads to LDS (rows past a chunk read as
// zero); prefix sums of g in fp64 log2 units (every decay factor is one exp2
// of an fp64 difference); each wave forms its share of the lower 16x16 blocks
// of K K^T and Q K^T with all its operands in registers, so the tiles' LDS
// space holds A, P and T afterwards; T's diagonal blocks by forward
// substitution with the rows of A in registers; its off-diagonal blocks one
// block diagonal at a time by fp32 MFMA block products; the fragments of W and
// P' from a bf16 copy of T.
template <int DK, int W, bool NORM>
__device__ __forceinline__ void gram_blocks(const bf16_t* sK, const bf16_t* sQ, const double* sGl, const float* sB,
                                            const float* sSk, const float* sSq, int l16, int lg, floatx4 (&ablk)[3],
                                            floatx4 (&pblk)[3]) {
    constexpr int NCH = DK / 8, NKD = DK / 32;
    // lower 16x16 blocks (bi, bj): KK^T takes entries W, W+4, ..; QK^T entries (W+2)%4, ..
    constexpr int BI[10] = {0, 1, 1, 2, 2, 2, 3, 3, 3, 3};
    constexpr int BJ[10] = {0, 0, 1, 0, 1, 2, 0, 1, 2, 3};
    constexpr int QW = (W + 2) % 4;
    constexpr int NA = W < 2 ? 3 : 2, NP = QW < 2 ? 3 : 2;
    auto swz = [](int r) { return ((4 * (r & 3)) | ((r >> 2) & 3)) & (NCH - 1); };
    auto kq = [&](int r, int cc) { return r * DK + (((cc >> 3) ^ swz(r)) << 3) + (cc & 7); };
    bf16x8 kf[4][NKD];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int kk = 0; kk < NKD; ++kk) kf[rb][kk] = *reinterpret_cast<const bf16x8*>(sK + kq(16 * rb + l16, 32 * kk + 8 * lg));
    bf16x8 qf[NP][NKD];
#pragma unroll
    for (int j = 0; j < NP; ++j)
#pragma unroll
        for (int kk = 0; kk < NKD; ++kk)
            qf[j][kk] = *reinterpret_cast<const bf16x8*>(sQ + kq(16 * BI[QW + 4 * j] + l16, 32 * kk + 8 * lg));
#pragma unroll
    for (int j = 0; j < NA; ++j) {
        const int bi = BI[W + 4 * j], bj = BJ[W + 4 * j];
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < NKD; ++kk) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[bi][kk], kf[bj][kk], acc, 0, 0, 0);
        const int i = 16 * bj + l16;
        const double gi = sGl[i];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int r = 16 * bi + 4 * lg + e;
            const float gam = __builtin_amdgcn_exp2f((float)(sGl[r] - gi));
            if constexpr (NORM) acc[e] *= sSk[r] * sSk[i];
            ablk[j][e] = r > i ? sB[r] * gam * acc[e] : 0.f;
        }
    }
#pragma unroll
    for (int j = 0; j < NP; ++j) {
        const int bi = BI[QW + 4 * j], bj = BJ[QW + 4 * j];
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < NKD; ++kk) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[j][kk], kf[bj][kk], acc, 0, 0, 0);
        const int i = 16 * bj + l16;
        const double gi = sGl[i];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int r = 16 * bi + 4 * lg + e;
            const float gam = __builtin_amdgcn_exp2f((float)(sGl[r] - gi));
            if constexpr (NORM) acc[e] *= sSq[r] * sSk[i];
            pblk[j][e] = r >= i ? gam * acc[e] : 0.f;
        }
    }
}

template <int DK, int W>
__device__ __forceinline__ void store_gram(float (*sA)[CH + 4], bf16_t (*sPb)[CH + 8], int l16, int lg,
                                           const floatx4 (&ablk)[3], const floatx4 (&pblk)[3]) {
    constexpr int BI[10] = {0, 1, 1, 2, 2, 2, 3, 3, 3, 3};
    constexpr int BJ[10] = {0, 0, 1, 0, 1, 2, 0, 1, 2, 3};
    constexpr int QW = (W + 2) % 4;
    constexpr int NA = W < 2 ? 3 : 2, NP = QW < 2 ? 3 : 2;
#pragma unroll
    for (int j = 0; j < NA; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) sA[16 * BI[W + 4 * j] + 4 * lg + e][16 * BJ[W + 4 * j] + l16] = ablk[j][e];
#pragma unroll
    for (int j = 0; j < NP; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) sPb[16 * BI[QW + 4 * j] + 4 * lg + e][16 * BJ[QW + 4 * j] + l16] = from_f<bf16_t>(pblk[j][e]);
}

// LDS of one chunk-terms work item: phase 1 holds the K and Q tiles; phase
// 2 reuses the space for A, T (fp32) and P (bf16), and T's bf16 copy over A
template <int DK> struct TermsLds {
    static constexpr int PA = CH + 4, PB = CH + 8;   // row pitches of the fp32 and bf16 64 x 64 matrices
    static constexpr int SZ_TILES = 2 * CH * DK * 2;
    static constexpr int SZ_MATS = 2 * CH * PA * 4 + CH * PB * 2;
    __attribute__((aligned(16))) char r0[SZ_TILES > SZ_MATS ? SZ_TILES : SZ_MATS];
    double sGl[CH];
    __attribute__((aligned(16))) float sB[CH];
    __attribute__((aligned(16))) float sD[CH];
    float sSk[CH], sSq[CH];   // reciprocal row lengths of K and Q (PRE_L2)
};

// Chunk terms of work item gi = chunk slot * H + head, by the 4 waves whose
// threads are tid = 0..255.  store = false computes without writing (a
// placeholder item that keeps a workgroup's two halves in step).  FUSED: every
// result is stored with cache-bypassing stores, then the slot's flag is set to
// the call's epoch; and the item's V rows, which only the chain reads, are
// copied into vsink (LDS nobody reads) so that they wait in L2 for the chain.
template <int DK, bool FUSED, bool NORM>
__device__ __forceinline__ void chunk_terms_bf16(const Params& p, const long gi, TermsLds<DK>& lds, const int tid,
                                                 const bool store, bf16_t* vsink = nullptr) {
    constexpr int NCH = DK / 8;     // 16-byte chunks per K/Q row
    constexpr int RPI = 64 / NCH;   // rows per 1 KB buffer load
    constexpr int TILE = CH * DK;
    constexpr int PA = TermsLds<DK>::PA, PB = TermsLds<DK>::PB;
    constexpr int AUX = FUSED ? 17 : 0;
    const int H = p.H;
    const int gc = (int)(gi / H), h = (int)(gi % H);
    int s;
    if (p.ragged) {
        if (gc >= tab(p.chunk_off, p.n_seq)) return;
        int lo = 0, hi = p.n_seq;
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (tab(p.chunk_off, mid) <= gc) lo = mid; else hi = mid;
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
    const long slot = (long)gc * H + h;

    char* r0 = lds.r0;
    double* sGl = lds.sGl;
    float* sB = lds.sB;
    float* sD = lds.sD;
    float* sSk = lds.sSk;
    float* sSq = lds.sSq;
    bf16_t* sK = reinterpret_cast<bf16_t*>(r0);
    bf16_t* sQ = sK + TILE;
    float(*sA)[PA] = reinterpret_cast<float(*)[PA]>(r0);
    float(*sTi)[PA] = reinterpret_cast<float(*)[PA]>(r0 + CH * PA * 4);
    bf16_t(*sPb)[PB] = reinterpret_cast<bf16_t(*)[PB]>(r0 + 2 * CH * PA * 4);
    bf16_t(*sTb)[PB] = reinterpret_cast<bf16_t(*)[PB]>(r0);

    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, lg = lane >> 4;
    auto swz = [](int r) { return ((4 * (r & 3)) | ((r >> 2) & 3)) & (NCH - 1); };

    {   // K and Q tiles straight into LDS; loads i = wave, wave + 4, ...
        const bf16_t* gk = reinterpret_cast<const bf16_t*>(p.k);
        const bf16_t* gq = reinterpret_cast<const bf16_t*>(p.q);
        const int HK = p.HK;   // q and k carry HK heads; this head reads key head h / G
        const long row0 = t0 * HK + h / p.G;
        const uint32_t bytes = (uint32_t)(((long)(n - 1) * HK + 1) * DK * 2);
        const auto rk = rsrc(gk + row0 * DK, bytes);
        const auto rq = rsrc(gq + row0 * DK, bytes);
        for (int i = wave; i < NCH; i += 4) {
            const int r = RPI * i + lane / NCH;
            const int off = (r * HK * DK + (((lane % NCH) ^ swz(r)) << 3)) * 2;
            bdma16(rk, sK + RPI * i * DK, off);
            bdma16(rq, sQ + RPI * i * DK, off);
        }
    }
    if (wave == 0) {
        // prefix sums of g in log2 units, fp64; padded rows: no decay, no write
        float gv = lane < n ? p.g[(t0 + lane) * H + h] : 0.f;
        float bv = lane < n ? p.beta[(t0 + lane) * H + h] : 0.f;
        if ((p.pre & PRE_GATES) && lane < n) {
            gv = gate_g(gv);
            bv = gate_beta(bv);
        }
        double x = (double)gv * 1.4426950408889634;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const double y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        const double xn = __shfl(x, 63, 64);
        const float dec = __builtin_amdgcn_exp2f((float)(xn - x));
        sGl[lane] = x;
        sB[lane] = bv;
        sD[lane] = dec;
        if (store) {
            const auto rg = rsrc(p.wsG + slot * GS, GS * 4);
            bstore4<AUX>(__builtin_amdgcn_exp2f((float)x), rg, lane * 4);
            bstore4<AUX>(dec, rg, (CH + lane) * 4);
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if constexpr (NORM) {
        // reciprocal row lengths: 4 lanes per row, each summing 4 of its 16-byte pieces (in any order)
        const int r = tid >> 2, part = tid & 3;
        float sk = 0.f, sq = 0.f;
#pragma unroll
        for (int j = 0; j < NCH / 4; ++j) {
            const bf16x8 a = *reinterpret_cast<const bf16x8*>(sK + r * DK + 8 * (NCH / 4 * part + j));
            const bf16x8 b = *reinterpret_cast<const bf16x8*>(sQ + r * DK + 8 * (NCH / 4 * part + j));
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                sk += (float)a[e] * (float)a[e];
                sq += (float)b[e] * (float)b[e];
            }
        }
        sk += __shfl_xor(sk, 1, 64);
        sk += __shfl_xor(sk, 2, 64);
        sq += __shfl_xor(sq, 1, 64);
        sq += __shfl_xor(sq, 2, 64);
        if (part == 0) {
            sSk[r] = r < n ? 1.f / sqrtf(sk + L2_EPS) : 0.f;
            sSq[r] = r < n ? 1.f / sqrtf(sq + L2_EPS) : 0.f;
        }
        __syncthreads();
        if (store && tid < CH) {   // the chain's decays for K S^T and Q S^T: gamma s_k, gamma s_q
            const auto rg = rsrc(p.wsG + slot * GS, GS * 4);
            const float gam = __builtin_amdgcn_exp2f((float)sGl[tid]);
            bstore4<AUX>(gam * sSk[tid], rg, (2 * CH + tid) * 4);
            bstore4<AUX>(gam * sSq[tid], rg, (3 * CH + tid) * 4);
        }
    }
    if constexpr (FUSED) {   // V rows of the item into L2 (waited for before the flag is set)
        const int DV = p.DV, vch = DV / 8, vrpi = 64 / vch;
        const auto rv = rsrc(reinterpret_cast<const bf16_t*>(p.v) + (t0 * H + h) * DV,
                             (uint32_t)(((long)(n - 1) * H + 1) * DV * 2));
        for (int i = wave; i < CH / vrpi; i += 4)
            bdma16(rv, vsink + i * 512, ((vrpi * i + lane / vch) * H * DV + (lane % vch) * 8) * 2);
    }

    // token-token blocks, all operands in registers
    floatx4 ablk[3], pblk[3];
    switch (wave) {
        case 0: gram_blocks<DK, 0, NORM>(sK, sQ, sGl, sB, sSk, sSq, l16, lg, ablk, pblk); break;
        case 1: gram_blocks<DK, 1, NORM>(sK, sQ, sGl, sB, sSk, sSq, l16, lg, ablk, pblk); break;
        case 2: gram_blocks<DK, 2, NORM>(sK, sQ, sGl, sB, sSk, sSq, l16, lg, ablk, pblk); break;
        default: gram_blocks<DK, 3, NORM>(sK, sQ, sGl, sB, sSk, sSq, l16, lg, ablk, pblk); break;
    }
    __syncthreads();   // every tile read done: A, P and T take the space over
    switch (wave) {
        case 0: store_gram<DK, 0>(sA, sPb, l16, lg, ablk, pblk); break;
        case 1: store_gram<DK, 1>(sA, sPb, l16, lg, ablk, pblk); break;
        case 2: store_gram<DK, 2>(sA, sPb, l16, lg, ablk, pblk); break;
        default: store_gram<DK, 3>(sA, sPb, l16, lg, ablk, pblk); break;
    }
    __syncthreads();

    // T = (I + A)^{-1}: diagonal blocks by forward substitution, one wave, lane =
    // 16 * block + column, A's block rows in registers.  The upper blocks of P
    // and T are never stored: their readers take them as zero.
    if (wave == 0) {
        const int b = lg;
        float a[16][16];
#pragma unroll
        for (int r = 1; r < 16; ++r)
#pragma unroll
            for (int q = 0; 4 * q < r; ++q) {
                const floatx4 v = *reinterpret_cast<const floatx4*>(&sA[16 * b + r][16 * b + 4 * q]);
#pragma unroll
                for (int t = 0; t < 4; ++t) a[r][4 * q + t] = v[t];
            }
        float x[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) x[r] = r == l16 ? 1.f : 0.f;
#pragma unroll
        for (int i = 0; i < 15; ++i)
#pragma unroll
            for (int r = i + 1; r < 16; ++r) x[r] -= a[r][i] * x[i];
#pragma unroll
        for (int r = 0; r < 16; ++r) sTi[16 * b + r][16 * b + l16] = x[r];
    }
    __syncthreads();
    // off-diagonal blocks, diagonal d: T_{b,b-d} = -T_bb sum_{m} A_bm T_{m,b-d}.
    // In MFMA step kk, lane group lg carries contraction index 4 lg + kk, so the
    // sum Z comes out of the accumulator exactly as the second product's B operand.
    for (int d = 1; d < 4; ++d) {
        if (wave < 4 - d) {
            const int j = wave, b = wave + d;
            floatx4 z = {0.f, 0.f, 0.f, 0.f};
            for (int m = j; m < b; ++m) {
                const floatx4 av = *reinterpret_cast<const floatx4*>(&sA[16 * b + l16][16 * m + 4 * lg]);
#pragma unroll
                for (int kk = 0; kk < 4; ++kk)
                    z = __builtin_amdgcn_mfma_f32_16x16x4f32(av[kk], sTi[16 * m + 4 * lg + kk][16 * j + l16], z, 0, 0, 0);
            }
            const floatx4 tv = *reinterpret_cast<const floatx4*>(&sTi[16 * b + l16][16 * b + 4 * lg]);
            floatx4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) t = __builtin_amdgcn_mfma_f32_16x16x4f32(tv[kk], z[kk], t, 0, 0, 0);
#pragma unroll
            for (int e = 0; e < 4; ++e) sTi[16 * b + 4 * lg + e][16 * j + l16] = -t[e];
        }
        __syncthreads();
    }
    for (int i = tid; i < CH * CH / 4; i += NT) {   // bf16 copy of T, zero above the diagonal blocks (A is no longer read)
        const int r = i / (CH / 4), c4 = 4 * (i % (CH / 4));
        floatx4 v = *reinterpret_cast<const floatx4*>(&sTi[r][c4]);
        if ((c4 >> 4) > (r >> 4)) v = floatx4{0.f, 0.f, 0.f, 0.f};
        *reinterpret_cast<bf16x4*>(&sTb[r][c4]) = __builtin_convertvector(v, bf16x4);
    }
    __syncthreads();

    const auto rW = rsrc(reinterpret_cast<bf16_t*>(p.wsT) + slot * tp_elems<bf16_t>(), tp_elems<bf16_t>() * 2);
    const auto rP = rsrc(reinterpret_cast<bf16_t*>(p.wsP) + slot * tp_elems<bf16_t>(), tp_elems<bf16_t>() * 2);
    for (int f = wave; f < NFRAG; f += 4) {
        const int mt = frag_mt(f), kk2 = frag_kk(f), r = 16 * mt + l16;
        // W fragment: D_r T[r][tau] beta_tau (times s_k,r with PRE_L2: the state update takes K unscaled)
        const float dr = NORM ? sD[r] * sSk[r] : sD[r];
        const floatx4 b0 = *reinterpret_cast<const floatx4*>(&sB[32 * kk2 + 4 * lg]);
        const floatx4 b1 = *reinterpret_cast<const floatx4*>(&sB[32 * kk2 + 16 + 4 * lg]);
        const floatx4 zero = {0.f, 0.f, 0.f, 0.f};   // blocks of T above the diagonal
        const floatx4 w0 = 2 * kk2 > mt ? zero : dr * b0 * *reinterpret_cast<const floatx4*>(&sTi[r][32 * kk2 + 4 * lg]);
        const floatx4 w1 =
            2 * kk2 + 1 > mt ? zero : dr * b1 * *reinterpret_cast<const floatx4*>(&sTi[r][32 * kk2 + 16 + 4 * lg]);
        if (store) bstore16<AUX>(pack_bf16(w0, w1), rW, (f * 64 + lane) * 16);
        // P' fragment from (T^T P^T) tiles (tau block 2 kk2 + hb, token block mt)
        floatx4 pt[2];
#pragma unroll
        for (int hb = 0; hb < 2; ++hb) {
            const int bt = 2 * kk2 + hb;
            pt[hb] = floatx4{0.f, 0.f, 0.f, 0.f};
            if (bt > mt) continue;   // above the diagonal: zero
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                const bf16_t* t0p = &sTb[32 * kk + 8 * lg + (l16 >> 2)][16 * bt + 4 * (l16 & 3)];
                const bf16x8 a = join4(lds_tr8(t0p), lds_tr8(t0p + 4 * PB));
                bf16x8 bb = *reinterpret_cast<const bf16x8*>(&sPb[16 * mt + l16][32 * kk + 8 * lg]);
                if (2 * kk + (lg >> 1) > mt) bb = bf16x8{};   // blocks of P above the diagonal
                pt[hb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bb, pt[hb], 0, 0, 0);
            }
            pt[hb] *= hb ? b1 : b0;
        }
        if (store) bstore16<AUX>(pack_bf16(pt[0], pt[1]), rP, (f * 64 + lane) * 16);
    }
    if constexpr (FUSED) {   // publish: every wave's stores are complete before the flag is set
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (tid == 0 && store && !p.withhold)   // (relaxed: see the flag poller of state_chain_bf16)
            __hip_atomic_store(&p.flags[slot], p.epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

template <int DK, bool NORM = false>
__global__ __launch_bounds__(NT, 3) void k_chunk_terms_bf16(Params p) {
    __shared__ TermsLds<DK> lds;
    chunk_terms_bf16<DK, false, NORM>(p, blockIdx.x, lds, threadIdx.x, true);
}

// One launch for the whole bf16 prefill: workgroups [0, npw) form chunk terms
// (two work items per workgroup, one per half of its waves, walking the items
// in chunk order), the rest are chain workgroups.  The chunk-terms workgroups
// are dispatched first and never wait, so the chain workgroups' waits end
// whatever number of workgroups the device holds at once.
template <int DK, bool SNAP = false, bool NORM = false>
__global__ __launch_bounds__(NT_CHAIN) __attribute__((amdgpu_waves_per_eu(1, 2))) void k_prefill_fused_bf16(Params p) {
    static_assert(NT_CHAIN == 2 * NT, "two work items per chunk-terms workgroup");
    __shared__ union Lds {
        ChainLds<DK> c;
        struct {
            TermsLds<DK> t;
            bf16_t vsink[CH * 128];
        } t[2];
    } lds;
    if ((int)blockIdx.x < p.npw) {
        const int half = __builtin_amdgcn_readfirstlane(threadIdx.x / NT);   // wave-uniform
        if (p.xcd_items) {
            // Dispatch deals workgroups to the 8 XCDs round-robin, so chain
            // workgroups of head h sit on XCD (npw + h) % 8.  Workgroup b forms
            // the items of heads h = (b - npw) mod 8 (+ 8 u), in chunk order, on
            // the XCD whose L2 then serves those chains.
            const int H = p.H, hu = H / 8, q = blockIdx.x / 8, nq = p.npw / 8;
            const int h0 = ((int)(blockIdx.x % 8) - p.npw % 8 + 8) % 8;
            const long items = (long)p.NC * p.n_seq * hu;   // per XCD
            for (long k = 2L * q; k < items; k += 2L * nq) {
                const long j = min(k + half, items - 1);
                const int c = (int)(j / ((long)p.n_seq * hu)), r = (int)((j / hu) % p.n_seq), u = (int)(j % hu);
                const long gi = ((long)r * p.NC + c) * H + h0 + 8 * u;
                chunk_terms_bf16<DK, true, NORM>(p, gi, lds.t[half].t, threadIdx.x % NT, k + half < items,
                                                 lds.t[half].vsink);
                __syncthreads();   // the next item reuses the LDS
            }
        } else {
            const long items = (long)(p.ragged ? tab(p.chunk_off, p.n_seq) : p.n_seq * p.NC) * p.H;
            for (long k = 2L * blockIdx.x; k < items; k += 2L * p.npw) {
                const long gi = item_slot(p, min(k + half, items - 1));   // both halves run every step together
                chunk_terms_bf16<DK, true, NORM>(p, gi, lds.t[half].t, threadIdx.x % NT, k + half < items,
                                                 lds.t[half].vsink);
                __syncthreads();   // the next item reuses the LDS
            }
        }
    } else {
        state_chain_bf16<DK, true, false, SNAP, NORM>(p, blockIdx.x - p.npw, lds.c);
    }
}

// ------------------------------------------------------------------ decode
// One token per sequence.  LPR lanes hold one state row as float4s; rows of S
// evolve independently: s_j <- alpha (s_j - beta (s_j.k) k) + beta v_j k.
template <typename IO, int DK>
__global__ __launch_bounds__(NT) void k_decode_step(const IO* __restrict__ q, const IO* __restrict__ k,
                                                    const IO* __restrict__ v, const float* __restrict__ g,
                                                    const float* __restrict__ beta, float* __restrict__ S,
                                                    IO* __restrict__ o, int H, int HK, int DV, int rows_per_wg,
                                                    float scale, int pre) {
    constexpr int LPR = DK / 4;        // lanes per row
    constexpr int RPP = NT / LPR;      // rows per pass of the workgroup
    const int bh = blockIdx.y;                                 // sequence * H + head
    const long bk = (long)(bh / H) * HK + (bh % H) / (H / HK);   // its key row: key head h / (H / HK)
    const int tid = threadIdx.x, sub = tid % LPR;
    float kv[4], qv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        kv[e] = to_f(k[bk * DK + 4 * sub + e]);
        qv[e] = to_f(q[bk * DK + 4 * sub + e]);
    }
    float sq = scale;
    if (pre & PRE_L2) {   // unit rows: the LPR lanes of a row hold all of k and q
        float kk = kv[0] * kv[0] + kv[1] * kv[1] + kv[2] * kv[2] + kv[3] * kv[3];
        float qq = qv[0] * qv[0] + qv[1] * qv[1] + qv[2] * qv[2] + qv[3] * qv[3];
#pragma unroll
        for (int m = LPR / 2; m >= 1; m >>= 1) {
            kk += __shfl_xor(kk, m, 64);
            qq += __shfl_xor(qq, m, 64);
        }
        const float sk = 1.f / sqrtf(kk + L2_EPS);
        sq *= 1.f / sqrtf(qq + L2_EPS);
#pragma unroll
        for (int e = 0; e < 4; ++e) kv[e] *= sk;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) qv[e] *= sq;
    const float a = expf((pre & PRE_GATES) ? gate_g(g[bh]) : g[bh]);
    const float b = (pre & PRE_GATES) ? gate_beta(beta[bh]) : beta[bh];
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

// ------------------------------------------------------------------ segment-parallel form
// The chunk map of section 3.2 is affine in the state: S_{c+1}^T = M_c S_c^T + N_c,
// so a run of chunks composes to S_end = S_start M_p + N_p (S orientation; M_p is
// the product of the chunks' M_c, transposed, and N_p what the run leaves from a
// zero state).  With each sequence cut at chunk boundaries into P segments of L
// chunks, all segments' chains run at once, twice, over the same chunk terms:
//   run 1: the true values, from S0 for segment 0 and from zero for the others.
//     It gives o for segment 0, for segment p the part o0 of o that leaves out
//     the state entering it, and the segment's N_p (its final state);
//   run 2: zero values from the identity (dk state rows).  Row i of its final
//     state is row i of M_p, and its output Y_t[i] = (e_i M_{p,t}) (scale q_t),
//     with M_{p,t} the map from the segment's start to token t, is what a unit
//     state row i adds to o_t.
// Rows of the state evolve independently of one another, so with X_p the state
// entering segment p:
//     X_1 = N_0,   X_{p+1} = X_p M_p + N_p,   o_t = o0_t + X_p Y_t  (t in segment p).
// Segments are packed as the sequences of a ragged call, so the chains and the
// chunk terms are the ragged kernels unchanged; the sequence table of that
// call has a closed form and is written directly.
struct SegParams {
    int nseq, P, L, T, NC, H, DV, DK;   // sequences; segments per sequence; chunks per segment; tokens and chunks per sequence
    int32_t* seq_start;  // the ragged call's sequence table over the nseq P segments (see Params):
    int32_t* seq_len;    //   token start and length, first chunk slot ([nseq P + 1]) and the
    int32_t* chunk_off;  //   chains' order
    int32_t* seq_perm;
    const float* S0;     // [nseq, H, DV, DK] or null (zeros)
    float* S0seg;        // [nseq P, H, DV, DK]: S0 for segment 0 of a sequence, zero for the others
    float* Iseg;         // [nseq P, H, DK, DK]: identity
    const float* N;      // run 1's final states [nseq P, H, DV, DK]
    const float* M;      // run 2's final states, transposed [nseq P, H, DK, DK] (bf16 for bf16 io)
    void* X;             // states entering each segment [nseq P, H, DV, DK], io (segment 0's unused)
    float* ST;           // [nseq, H, DV, DK] or null
    const void* Y;       // run 2's outputs [nseq T, H, DK] io
    void* o;             // [nseq T, H, DV] io
};

// Segment table and the two runs' initial states: workgroup row y is segment
// y (row nseq P only writes the table's end).
template <int DK>
__global__ __launch_bounds__(NT) void k_segment_prep(SegParams sp) {
    const int seg = blockIdx.y, nseg = sp.nseq * sp.P;
    const int i = blockIdx.x * NT + threadIdx.x;   // float4 within one segment's matrices
    if (i == 0) {   // segment p of sequence b: chunks [p L, min((p + 1) L, NC)) of the sequence
        const int b = seg / sp.P, p = seg % sp.P;
        sp.chunk_off[seg] = b * sp.NC + min(p * sp.L, sp.NC);
        if (seg < nseg) {
            const long t0 = std::min((long)p * sp.L * CH, (long)sp.T), t1 = std::min((long)(p + 1) * sp.L * CH, (long)sp.T);
            sp.seq_start[seg] = (int32_t)((long)b * sp.T + t0);
            sp.seq_len[seg] = (int32_t)(t1 - t0);
            sp.seq_perm[seg] = seg;
        }
    }
    if (seg >= nseg) return;
    const int mat4 = sp.H * sp.DV * (DK / 4), id4 = sp.H * DK * (DK / 4);
    if (i < mat4) {
        floatx4 x = {0.f, 0.f, 0.f, 0.f};
        if (sp.S0 && seg % sp.P == 0) x = reinterpret_cast<const floatx4*>(sp.S0)[(long)(seg / sp.P) * mat4 + i];
        reinterpret_cast<floatx4*>(sp.S0seg)[(long)seg * mat4 + i] = x;
    }
    if (i < id4) {
        const int r = (i / (DK / 4)) % DK, c0 = (i % (DK / 4)) * 4;
        floatx4 x;
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = c0 + e == r ? 1.f : 0.f;
        reinterpret_cast<floatx4*>(sp.Iseg)[(long)seg * id4 + i] = x;
    }
}

// The scan over segments: one workgroup per (sequence, head, 16 state rows);
// rows of X never mix, so the workgroups are independent.  X (16 x DK, fp32)
// sits in LDS; wave w forms column tile w of X M_p + N_p on MFMA (bf16
// operands for bf16 io, fp32 for fp32 io) and writes X_p out in io precision
// for the output pass.  M_p arrives transposed, so a lane's B fragment is one
// contiguous run of a row of M_p^T.  M_p and N_p do not depend on X: a ring of R
// register slots keeps the next R segments' fragments in flight, with the
// segment loop unrolled by R so slots are never copied (a copy would wait for
// its load), and the barriers order LDS only.
template <typename IO, int DK>
__global__ __launch_bounds__(DK * 4) void k_segment_scan(SegParams sp) {
    constexpr bool BF = sizeof(IO) == 2;
    constexpr int NTH = DK * 4;   // DK / 16 waves
    constexpr int NF = DK / 16;   // 16-byte loads of M_p^T per lane and segment (bf16: DK / 32)
    constexpr int R = 4;
    __shared__ __attribute__((aligned(16))) float sX[2][SL][DK + 4];
    const int H = sp.H, DV = sp.DV, nsl = DV / SL, P = sp.P;
    // Dispatch deals workgroups to the 8 XCDs round-robin: workgroup w runs on
    // XCD w % 8.  All slices of one (sequence, head) go to one XCD, so its L2
    // serves the M_p and N_p that every slice reads; the grid is padded to
    // whole XCD rounds and the spare workgroups exit.
    const int xcd = blockIdx.x % 8, k = blockIdx.x / 8;
    const int unit = (k / nsl) * 8 + xcd, js = k % nsl;
    if (unit >= sp.nseq * H) return;
    const int h = unit % H, b = unit / H;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), l16 = lane & 15, lg = lane >> 4;
    const int col = 16 * wave + l16;
    const long mat = (long)DV * DK;
    auto rows_at = [&](int seg) { return ((long)seg * H + h) * mat + (long)js * SL * DK; };
    // contraction index of element e of lane group lg in step j: fp32: (DK/4) lg + 4 j + e;
    // bf16 (steps of 8 = two float4s): 32 (j/2) + 8 lg + 4 (j%2) + e
    auto koff = [&](int j) { return BF ? 32 * (j >> 1) + 8 * lg + 4 * (j & 1) : (DK / 4) * lg + 4 * j; };
    typedef typename std::conditional<BF, bf16x8, floatx4>::type MF;
    constexpr int NM = BF ? DK / 32 : NF;
    MF m[R][NM];
    floatx4 nf[R];
    {
        const float* n0 = sp.N + rows_at(b * P);
        for (int i = tid; i < SL * DK; i += NTH) sX[0][i / DK][i % DK] = n0[i];
    }
    // loads never branch (past the last segment they repeat it), so the
    // compiler's wait counts stay exact across the unrolled loop
    auto load = [&](int p, MF (&mr)[NM], floatx4& n) {
        p = min(p, P - 1);
        const long mt = ((long)(b * P + p) * H + h) * DK * DK + (long)col * DK;   // row col of M_p^T
        if constexpr (BF) {
            const bf16_t* Mt = reinterpret_cast<const bf16_t*>(sp.M) + mt;
#pragma unroll
            for (int kk = 0; kk < NM; ++kk) mr[kk] = *reinterpret_cast<const bf16x8*>(Mt + koff(2 * kk));
        } else {
            const float* Mt = sp.M + mt;
#pragma unroll
            for (int j = 0; j < NF; ++j) mr[j] = *reinterpret_cast<const floatx4*>(Mt + koff(j));
        }
        const float* Np = sp.N + rows_at(b * P + p);
#pragma unroll
        for (int e = 0; e < 4; ++e) n[e] = Np[(4 * lg + e) * DK + col];
    };
#pragma unroll
    for (int d = 0; d < R; ++d) load(1 + d, m[d], nf[d]);
    lds_barrier();
    int cur = 0;
    auto step = [&](int p, auto D) {
        constexpr int d = decltype(D)::value;
        {   // X_p out: one float4 per thread (a fixed count keeps the load counters exact)
            static_assert(SL * DK == 4 * NTH, "one float4 of X per thread");
            const int r = 4 * tid / DK, cc = 4 * tid % DK;
            const floatx4 x = f4(&sX[cur][r][cc]);
            IO* xo = reinterpret_cast<IO*>(sp.X) + rows_at(b * P + p) + 4 * tid;
            if constexpr (BF) {
                const uint2 u = {(uint32_t)from_f<bf16_t>(x[0]) | ((uint32_t)from_f<bf16_t>(x[1]) << 16),
                                 (uint32_t)from_f<bf16_t>(x[2]) | ((uint32_t)from_f<bf16_t>(x[3]) << 16)};
                *reinterpret_cast<uint2*>(xo) = u;
            } else {
                *reinterpret_cast<floatx4*>(xo) = x;
            }
        }
        floatx4 acc = nf[d];
        if constexpr (BF) {
#pragma unroll
            for (int kk = 0; kk < DK / 32; ++kk) {
                const bf16x8 a = pack_bf16(f4(&sX[cur][l16][koff(2 * kk)]), f4(&sX[cur][l16][koff(2 * kk + 1)]));
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, m[d][kk], acc, 0, 0, 0);
            }
        } else {
#pragma unroll
            for (int j = 0; j < NF; ++j) {
                const floatx4 a = f4(&sX[cur][l16][koff(j)]);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], m[d][j][e], acc, 0, 0, 0);
            }
        }
        // acc[e]: row 4 lg + e, column col of X_p M_p + N_p
#pragma unroll
        for (int e = 0; e < 4; ++e) sX[cur ^ 1][4 * lg + e][col] = acc[e];
        load(p + R, m[d], nf[d]);
        lds_barrier();
        cur ^= 1;
    };
    static_assert(R == 4, "the loop below is unrolled by 4");
    int p0 = 1;
    for (; p0 + R <= P; p0 += R) {
        step(p0, Ic<0>{});
        step(p0 + 1, Ic<1>{});
        step(p0 + 2, Ic<2>{});
        step(p0 + 3, Ic<3>{});
    }
    if (p0 < P) step(p0, Ic<0>{});
    if (p0 + 1 < P) step(p0 + 1, Ic<1>{});
    if (p0 + 2 < P) step(p0 + 2, Ic<2>{});
    if (sp.ST) {
        float* st = sp.ST + ((long)b * H + h) * mat + (long)js * SL * DK;
        for (int i = tid; i < SL * DK; i += NTH) st[i] = sX[cur][i / DK][i % DK];
    }
}

// o_t += X_p Y_t for the chunks of segments p >= 1: one workgroup of 8 waves
// per (sequence, segment, head, pair of chunks), X_p (io precision) staged in
// LDS.  Wave w takes tokens 16 (w%4)..+15 of the pair's chunk w/4 and forms
// (X_p Y^T) tile by tile, so a lane ends up with 4 consecutive value channels
// of one token.  Its Y fragments and the o values it updates are loaded
// before the staging.
constexpr int NT_CORR = 512;
template <typename IO, int DK>
__global__ __launch_bounds__(NT_CORR) void k_segment_correct(SegParams sp) {
    constexpr bool BF = sizeof(IO) == 2;
    constexpr int PADX = BF ? 8 : 4;
    constexpr int DVM = 128;                     // largest value width
    constexpr int NKB = BF ? DK / 32 : DK / 4;   // contraction steps
    constexpr int VEC = 16 / sizeof(IO);         // elements per 16-byte load
    __shared__ __attribute__((aligned(16))) IO sXp[DVM][DK + PADX];
    const int H = sp.H, DV = sp.DV, npair = (sp.L + 1) / 2;
    // all workgroups of one (sequence, segment, head) on one XCD (workgroup w runs
    // on XCD w % 8), whose L2 then serves their reads of X_p; spare ones exit
    const int xcd = blockIdx.x % 8, k = blockIdx.x / 8;
    const long unit = (long)(k / npair) * 8 + xcd;
    if (unit >= (long)sp.nseq * (sp.P - 1) * H) return;
    const int q = k % npair;
    const int h = (int)(unit % H);
    const int p = 1 + (int)((unit / H) % (sp.P - 1));
    const int b = (int)(unit / ((long)H * (sp.P - 1)));
    const int seg = b * sp.P + p;
    const int c_end = min((p + 1) * sp.L, sp.NC);   // one past the segment's last chunk
    const int c0 = p * sp.L + 2 * q;
    if (c0 >= c_end) return;                        // workgroup-uniform
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), l16 = lane & 15, lg = lane >> 4;
    const int c = c0 + wave / 4;
    const long t_end = (long)b * sp.T + sp.T;       // one past the sequence's last token
    const long t = (long)b * sp.T + (long)c * CH + 16 * (wave % 4) + l16;   // this lane's token
    const bool live = c < c_end && t < t_end;
    const long tb = live ? t : (long)b * sp.T;      // a valid row for the Y reads of idle lanes
    const IO* y = reinterpret_cast<const IO*>(sp.Y) + (tb * H + h) * DK;
    IO* o = reinterpret_cast<IO*>(sp.o) + (t * H + h) * DV + 4 * lg;
    typedef typename std::conditional<BF, bf16x8, float>::type YF;
    YF yb[NKB];
#pragma unroll
    for (int kk = 0; kk < NKB; ++kk) {
        if constexpr (BF) yb[kk] = *reinterpret_cast<const bf16x8*>(y + 32 * kk + 8 * lg);
        else yb[kk] = y[4 * kk + lg];
    }
    floatx4 ov[DVM / 16];
#pragma unroll
    for (int n = 0; n < DVM / 16; ++n) {
        ov[n] = floatx4{0.f, 0.f, 0.f, 0.f};
        if (live && n < DV / 16) {
            if constexpr (BF) {
                const uint2 u = *reinterpret_cast<const uint2*>(o + 16 * n);
                ov[n] = floatx4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                                __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u)};
            } else {
                ov[n] = *reinterpret_cast<const floatx4*>(o + 16 * n);
            }
        }
    }
    const IO* xp = reinterpret_cast<const IO*>(sp.X) + ((long)seg * H + h) * DV * DK;
#pragma unroll
    for (int j = 0; j < DVM * DK / VEC / NT_CORR; ++j) {
        const int i = tid + NT_CORR * j;
        if (i < DV * DK / VEC) {
            const int r = (VEC * i) / DK, cc = (VEC * i) % DK;
            *reinterpret_cast<uint4*>(&sXp[r][cc]) = reinterpret_cast<const uint4*>(xp)[i];
        }
    }
    __syncthreads();
#pragma unroll
    for (int n = 0; n < DVM / 16; ++n) {
        if (n >= DV / 16) break;
        floatx4 acc = ov[n];
#pragma unroll
        for (int kk = 0; kk < NKB; ++kk) {
            if constexpr (BF)
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    *reinterpret_cast<const bf16x8*>(&sXp[16 * n + l16][32 * kk + 8 * lg]), yb[kk], acc, 0, 0, 0);
            else
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(sXp[16 * n + l16][4 * kk + lg], yb[kk], acc, 0, 0, 0);
        }
        // acc[e]: value channel 16 n + 4 lg + e of this lane's token
        if (live) {
            if constexpr (BF) {
                const uint2 u = {(uint32_t)from_f<bf16_t>(acc[0]) | ((uint32_t)from_f<bf16_t>(acc[1]) << 16),
                                 (uint32_t)from_f<bf16_t>(acc[2]) | ((uint32_t)from_f<bf16_t>(acc[3]) << 16)};
                *reinterpret_cast<uint2*>(o + 16 * n) = u;
            } else {
                *reinterpret_cast<floatx4*>(o + 16 * n) = acc;
            }
        }
    }
}

// Paired chain launch: workgroups [0, first) run the problem in p, the rest the
// same chunks with another value tensor, width, initial and final states and
// output (the identity run of the segment-parallel form).
struct ChainAlt {
    const void* v;
    const float* S0;
    void* o;
    float* ST;
    int st_t;
    int DV;
    int first;
};

template <int DK, bool NORM = false>
__global__ __launch_bounds__(NT_CHAIN) __attribute__((amdgpu_waves_per_eu(1, 2))) void k_state_chain_pair_bf16(Params p,
                                                                                                         ChainAlt a) {
    __shared__ ChainLds<DK> lds;
    const int bid = blockIdx.x;
    if (bid >= a.first) {
        p.v = a.v; p.S0 = a.S0; p.o = a.o; p.ST = a.ST; p.st_t = a.st_t; p.DV = a.DV;
        state_chain_bf16<DK, false, true, false, NORM>(p, bid - a.first, lds);
    } else {
        state_chain_bf16<DK, false, false, false, NORM>(p, bid, lds);
    }
}

template <int DK>
__global__ __launch_bounds__(NT_CHAIN) __attribute__((amdgpu_waves_per_eu(1, 2))) void k_state_chain_pair(Params p, ChainAlt a) {
    __shared__ F32ChainLds<DK> lds;
    int bid = blockIdx.x;
    if (bid >= a.first) { p.v = a.v; p.S0 = a.S0; p.o = a.o; p.ST = a.ST; p.st_t = a.st_t; p.DV = a.DV; bid -= a.first; }
    state_chain_f32<DK>(p, bid, lds);
}

// ------------------------------------------------------------------ causal attention prefill
// The backbone's softmax-attention layers over a prompt (section 5: scores Q K^T
// per head, a causal softmax, then P V; grouped query heads share a key/value
// head): per (sequence, head h),
//     o_i = sum_{j <= i} softmax_j(scale q_i . k_j) v_j,   key/value head h / (H / H_kv).
// One workgroup per (sequence, head, block of AQ queries): 8 waves of one 16-query
// tile, or 4 waves of two (QT); blocks of AKB keys and values stream through a
// double-buffered LDS ring (16-byte chunks XOR-swizzled by row) up to the causal
// diagonal.  Per key block a wave forms S^T = K Q^T for each of its query tiles
// (Q^T operands held in registers; each K operand read serves all the tiles), the
// running softmax of each query column in fp32 (the block maximum across the lane
// groups by shuffles), and O^T += V^T P^T: the exponentiated S^T accumulators are
// the B operand as they stand (contraction over keys in the order
// 32 kk + 16 (j / 4) + 4 lg + j % 4), and the V^T operands come from transpose LDS
// reads in that order.  The full score matrix never exists; the work skips key
// blocks past a wave's last query.
constexpr int AQ = 128, AKB = 64, NT_ATT = 512;

struct AttnParams {
    const bf16_t* q;
    const bf16_t* k;
    const bf16_t* v;
    bf16_t* o;
    int B, T, H, HKV;
    int nqb;            // dense: query blocks per sequence; packed: blocks of the grid per head (an upper bound)
    const int32_t* cu;  // packed sequences: offsets [n_seq + 1] (device), or null
    int n_seq;
    float scale_log2;   // scale * log2(e)
};

template <int DH> struct AttnLds {
    bf16_t k[2][AKB * DH];
    bf16_t v[2][AKB * DH];
};

template <int DH, int QT>
__global__ __launch_bounds__(NT_ATT / QT) __attribute__((amdgpu_waves_per_eu(4 / QT))) void k_attn_causal(AttnParams p) {
    constexpr int NW = NT_ATT / 64 / QT;   // waves; each holds QT tiles of 16 queries
    constexpr int NCH = DH / 8;         // 16-byte chunks per row
    constexpr int RPI = 64 / NCH;       // rows per 1 KB copy
    constexpr int NKB = DH / 32;        // contraction blocks over the head dimension
    constexpr int NDT = DH / 16;        // 16-row tiles of O^T
    constexpr int NCP = 2 * AKB / RPI;  // 1 KB copies per key block (K and V)
    __shared__ AttnLds<DH> lds;
    const int BH = p.B * p.H;
    int qb = p.nqb - 1 - (int)(blockIdx.x / BH);   // blocks with the most keys first
    const int bh = (int)(blockIdx.x % BH);
    const int b = bh / p.H, h = bh % p.H, hk = h / (p.H / p.HKV);
    // the wave index as a scalar: the branches on it below (masking, skipped blocks,
    // K or V copies) are then scalar branches
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, lg = lane >> 4;
    long seq0 = (long)b * p.T;   // first row of this workgroup's sequence
    int T = p.T;                 // its length
    if (p.cu) {
        // packed sequences (B = 1): grid block qb (counted from the top) is block j of sequence s, where the
        // sequences' blocks are numbered consecutively, each sequence's last block first.  Offsets outside the
        // contract are clamped into a nondecreasing partition of [0, p.T], so every access stays in bounds.
        int prev = 0, before = 0, s = 0;
        int found = -1;
        for (; s < p.n_seq; ++s) {
            const int next = min(max(tab(p.cu, s + 1), prev), p.T);
            const int nb = (next - prev + AQ - 1) / AQ;
            const int r = p.nqb - 1 - qb;   // rank of this block in that numbering
            if (r < before + nb) {
                found = nb - 1 - (r - before);
                seq0 = prev;
                T = next - prev;
                break;
            }
            before += nb;
            prev = next;
        }
        if (found < 0) return;   // past the last block (the grid is an upper bound)
        qb = found;
    }
    const int q0 = qb * AQ, qw = q0 + 16 * QT * wave;   // the workgroup's and this wave's first query
    const long rsq = (long)p.H * DH, rsk = (long)p.HKV * DH;   // row strides (elements)
    const bf16_t* qbase = p.q + (seq0 * p.H + h) * DH;
    const bf16_t* kbase = p.k + (seq0 * p.HKV + hk) * DH;
    const bf16_t* vbase = p.v + (seq0 * p.HKV + hk) * DH;
    // 16-byte chunk c of row r sits at chunk c ^ swz(r).  Both reads below are free of bank conflicts with it: the
    // K read's 16 rows in a group of 16 lanes, and the V read's 8 rows x 2 chunks in a group of 32 lanes (row bit 2
    // lands on chunk bit 1, which neither the row's low bits nor the chunk pair use).  At d = 64 two rows share
    // the 64 banks, so row bit 0 is left to the row stride.
    auto swz = [](int r) {
        return NCH == 16 ? (4 * (r & 3)) | (2 * ((r >> 2) & 1)) | ((r >> 3) & 1)
                         : (4 * ((r >> 1) & 1)) | (2 * ((r >> 2) & 1)) | ((r >> 3) & 1);
    };
    auto kq = [swz](int r, int cc) { return r * DH + (((cc >> 3) ^ swz(r)) << 3) + (cc & 7); };
    // descriptor over rows [r0, min(r0 + n, T)) of a [T][heads][DH] tensor; rows past T read as zeros
    auto rows_rsrc = [&](const bf16_t* base, long rs, int r0, int n) {
        const int m = min(n, T - r0);
        return rsrc(base + (long)r0 * rs, m > 0 ? (uint32_t)(((long)(m - 1) * rs + DH) * 2) : 0u);
    };

    // Q^T operands: lane holds q[qw + 16 u + l16][32 kb + 8 lg .. + 7] for query tile u
    bf16x8 qf[QT][NKB];
    {
        const auto rq = rows_rsrc(qbase, rsq, qw, 16 * QT);
#pragma unroll
        for (int u = 0; u < QT; ++u)
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) qf[u][kb] = bload16(rq, (int)(((16 * u + l16) * rsq + 32 * kb + 8 * lg) * 2));
    }
    // copies of key block j into ring slot j & 1: copy c < NCP / 2 is K rows RPI c .., the rest V
    const int nkb = min((T + AKB - 1) / AKB, (q0 + AQ) / AKB);
    auto issue = [&](int j) {
        const int kb0 = j * AKB, sl = j & 1;
        const auto rk = rows_rsrc(kbase, rsk, kb0, AKB);
        const auto rv = rows_rsrc(vbase, rsk, kb0, AKB);
#pragma unroll
        for (int c = wave; c < NCP; c += NW) {
            const int cc = c % (NCP / 2), r = RPI * cc + lane / NCH;
            const int off = (int)((r * rsk + (((lane % NCH) ^ swz(r)) << 3)) * 2);
            if (c < NCP / 2) bdma16(rk, &lds.k[sl][RPI * cc * DH], off);
            else bdma16(rv, &lds.v[sl][RPI * cc * DH], off);
        }
    };
    // Running softmax per query in log2 units.  m is a reference at most RESLACK below
    // the largest scaled score seen (it moves only when a block exceeds it by more:
    // the weights 2^(x - m) stay below 2^RESLACK, and O and the weight sum are
    // rescaled only then).  The weight sum is one more product tile, ones times the
    // bf16 weights, so it sums exactly the weights the products with V use: every
    // entry of lsum is the sum of this lane's query.
    constexpr float RESLACK = 8.f;
    const float sl2 = p.scale_log2;
    const floatx4 one4 = {1.f, 1.f, 1.f, 1.f};
    const bf16x8 ones = pack_bf16(one4, one4);
    float m[QT];
    floatx4 lsum[QT], oacc[QT][NDT];
#pragma unroll
    for (int u = 0; u < QT; ++u) {
        m[u] = -INFINITY;
        lsum[u] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < NDT; ++t) oacc[u][t] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
    // key block j in ring slot SL = j & 1 (a constant: the loop below is unrolled by two,
    // so the LDS addresses are this lane's offsets plus immediates)
    auto block = [&](const int j, auto SLOT) {
        constexpr int SL = decltype(SLOT)::value;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's copies of block j
        lds_barrier();                                       // everyone's; slot (j + 1) & 1 no longer read
        if (j + 1 < nkb) issue(j + 1);
        const int kb0 = j * AKB;
        if (kb0 > qw + 16 * QT - 1) return;   // every key of the block follows this wave's queries
        const bf16_t* sk = lds.k[SL];
        const bf16_t* sv = lds.v[SL];
        floatx4 st[QT][4];   // S^T of query tile u: keys 16 t + 4 lg + e, query l16
#pragma unroll
        for (int u = 0; u < QT; ++u)
#pragma unroll
            for (int t = 0; t < 4; ++t) st[u][t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                const bf16x8 ka = *reinterpret_cast<const bf16x8*>(&sk[kq(16 * t + l16, 32 * kb + 8 * lg)]);
#pragma unroll
                for (int u = 0; u < QT; ++u) st[u][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qf[u][kb], st[u][t], 0, 0, 0);
            }
        bf16x8 pf[QT][2];
#pragma unroll
        for (int u = 0; u < QT; ++u) {
            const int qt0 = qw + 16 * u;   // the tile's first query
            // some key of the block is masked for this tile (wave-uniform)
            const bool diag = kb0 + AKB - 1 > qt0 || kb0 + AKB > T;
            // bm: the block's largest scaled score of this lane's query; the weights are
            // 2^(fs x - m).  Blocks with no masked key and a scale >= 0 take the largest
            // raw score times the scale (fs = scale); otherwise the scores are scaled and
            // masked first (fs = 1).
            float bm, fs;
            if (!diag && sl2 >= 0.f) {
                bm = st[u][0][0];
#pragma unroll
                for (int t = 0; t < 4; ++t)
#pragma unroll
                    for (int e = 0; e < 4; ++e) bm = fmaxf(bm, st[u][t][e]);
                bm = fmaxf(bm, __shfl_xor(bm, 16, 64));
                bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
                bm *= sl2;
                fs = sl2;
            } else {
                const int qi = qt0 + l16;
                bm = -INFINITY;
#pragma unroll
                for (int t = 0; t < 4; ++t)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int kj = kb0 + 16 * t + 4 * lg + e;
                        const float x = (kj > qi || kj >= T) ? -INFINITY : st[u][t][e] * sl2;
                        st[u][t][e] = x;
                        bm = fmaxf(bm, x);
                    }
                bm = fmaxf(bm, __shfl_xor(bm, 16, 64));
                bm = fmaxf(bm, __shfl_xor(bm, 32, 64));
                fs = 1.f;
            }
            // the first block holds key 0 <= every query, so m is finite from then on; a
            // later block may mask every key of a query (bm = -inf): m stays
            const bool up = bm > m[u] + RESLACK;
            if (__builtin_amdgcn_ballot_w64(up)) {
                const float mn = up ? bm : m[u];
                const float alpha = __builtin_amdgcn_exp2f(m[u] - mn);   // 1 where m stays; 0 at the first block
#pragma unroll
                for (int t = 0; t < NDT; ++t) oacc[u][t] *= alpha;
                lsum[u] *= alpha;
                m[u] = mn;
            }
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int e = 0; e < 4; ++e) st[u][t][e] = __builtin_amdgcn_exp2f(__builtin_fmaf(st[u][t][e], fs, -m[u]));
            pf[u][0] = pack_bf16(st[u][0], st[u][1]);
            pf[u][1] = pack_bf16(st[u][2], st[u][3]);
            lsum[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[u][0], lsum[u], 0, 0, 0);
            lsum[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[u][1], lsum[u], 0, 0, 0);
        }
#pragma unroll
        for (int t = 0; t < NDT; ++t) {
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                const int r = 32 * kk + 4 * lg + (l16 >> 2), c = 16 * t + 4 * (l16 & 3);
                const bf16x8 va = join4(lds_tr8(&sv[kq(r, c)]), lds_tr8(&sv[kq(r + 16, c)]));
#pragma unroll
                for (int u = 0; u < QT; ++u) oacc[u][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pf[u][kk], oacc[u][t], 0, 0, 0);
            }
        }
    };
    if (nkb > 0) issue(0);
    for (int j = 0; j < nkb; j += 2) {
        block(j, Ic<0>{});
        if (j + 1 < nkb) block(j + 1, Ic<1>{});
    }
    // o[qw + 16 u + l16][16 t + 4 lg + e] = O^T / (weight sum)
#pragma unroll
    for (int u = 0; u < QT; ++u) {
        const int qi = qw + 16 * u + l16;
        if (qi < T) {
            const float inv = 1.f / lsum[u][0];
            bf16_t* orow = p.o + ((seq0 + qi) * p.H + h) * DH;
#pragma unroll
            for (int t = 0; t < NDT; ++t) {
                const floatx4 ov = oacc[u][t] * inv;
                *reinterpret_cast<bf16x4*>(orow + 16 * t + 4 * lg) = __builtin_convertvector(ov, bf16x4);
            }
        }
    }
}

#include "wide.hip"
#include "generic.hip"

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
    size_t meta, G, T, P, F, KQ, total;
};

// Workspace layout; returns false for arguments that are out of range.
bool ws_layout(int B, int T, int H, int dk, int dv, int n_seqs, int io, Layout* L) {
    (void)dv;
    const size_t esz = io == GDN_BF16 ? 2 : 4;
    const long cpt = ((long)T + CH - 1) / CH;
    L->slots = n_seqs > 0 ? cpt + n_seqs : (long)B * cpt;
    if (L->slots * (long)H > (1L << 24)) return false;
    const size_t per = (size_t)L->slots * H;
    if (per == 0) {   // no chunk: nothing to keep (not even the status word)
        L->meta = L->G = L->T = L->P = L->F = L->KQ = L->total = 0;
        return true;
    }
    L->meta = 256;   // bytes [0, 8): the status word (gdn_workspace_status)
    L->G = L->meta + (n_seqs > 0 ? round_up(((size_t)4 * (n_seqs + 1) + 2 * (size_t)(cpt + 2)) * sizeof(int32_t), 256) : 0);
    L->T = L->G + round_up(per * GS * sizeof(float), 256);
    const size_t tp = io == GDN_BF16 ? tp_elems<bf16_t>() : tp_elems<float>();
    L->P = L->T + round_up(per * tp * esz, 256);
    L->F = L->P + round_up(per * tp * esz, 256);
    L->KQ = L->F + (io == GDN_BF16 ? round_up(per * sizeof(uint64_t), 256) : 0);
    // fp32 io: K and Q of every (chunk slot, head) as high and low bf16 parts, in the chain's LDS order
    L->total = L->KQ + (io == GDN_BF16 ? 0 : round_up(per * 4 * CH * (size_t)dk * sizeof(bf16_t), 256));
    return true;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Chunk lengths and workspace of the generic path (chunk != 64): the status word,
// the ragged table, and per (chunk slot, head) 4 C floats (gamma, D, s_k, s_q)
// and two C x C fp32 matrices (A then W; P then P').
bool gen_chunk(int chunk) { return chunk == 16 || chunk == 32 || chunk == 128; }

bool gen_layout(int B, int T, int H, int C, int n_seqs, Layout* L) {
    const long cpt = ((long)T + C - 1) / C;
    L->slots = n_seqs > 0 ? cpt + n_seqs : (long)B * cpt;
    if (L->slots * (long)H > (1L << 24)) return false;
    const size_t per = (size_t)L->slots * H;
    if (per == 0) {
        L->meta = L->G = L->T = L->P = L->F = L->KQ = L->total = 0;
        return true;
    }
    L->meta = 256;
    L->G = L->meta + (n_seqs > 0 ? round_up(((size_t)4 * (n_seqs + 1) + 2 * (size_t)(cpt + 2)) * sizeof(int32_t), 256) : 0);
    L->T = L->G + round_up(per * 4 * C * sizeof(float), 256);
    L->P = L->T + round_up(per * C * C * sizeof(float), 256);
    L->F = L->P + round_up(per * C * C * sizeof(float), 256);
    L->KQ = L->total = L->F;
    return true;
}

template <typename IO, int C, int DK>
void launch_generic_c(const Params& p, long slots, hipStream_t st) {
    if (p.ragged)
        hipLaunchKernelGGL(k_ragged_setup, dim3(1), dim3(NSET), 0, st, p.cu, p.n_seq, p.T, p.seq_start, p.seq_len,
                           p.chunk_off, p.seq_perm, p.cprefix, p.cprefix + (p.cpt + 2), p.cpt, C);
    if (slots > 0 && p.T > 0) {
        hipLaunchKernelGGL((k_gen_gram<IO, C, DK>), dim3((unsigned)(slots * p.H)), dim3(GEN_NT), 0, st, p);
        hipLaunchKernelGGL((k_gen_solve<C>), dim3((unsigned)(slots * p.H)), dim3(GEN_NT), 0, st, p);
    }
    hipLaunchKernelGGL((k_gen_chain<IO, C, DK>), dim3((unsigned)(p.n_seq * p.H * (p.DV / GEN_RS))), dim3(GEN_NT), 0, st, p);
}

template <typename IO, int DK>
void launch_generic(const Params& p, long slots, hipStream_t st) {
    switch (p.C) {
        case 16: launch_generic_c<IO, 16, DK>(p, slots, st); break;
        case 32: launch_generic_c<IO, 32, DK>(p, slots, st); break;
        default: launch_generic_c<IO, 128, DK>(p, slots, st); break;
    }
}

// The device a stream's work runs on (NULL: the current device); -1 when there is none.
int stream_device(hipStream_t st) {
    int dev = -1;
    if (st == nullptr || hipStreamGetDevice(st, &dev) != hipSuccess) {
        (void)hipGetLastError();
        if (hipGetDevice(&dev) != hipSuccess) {
            (void)hipGetLastError();
            return -1;
        }
    }
    return dev >= 0 && dev < 64 ? dev : -1;
}

// Compute units of the device a stream's work runs on (cached per device).
int stream_cus(hipStream_t st) {
    static std::atomic<int> cached[64];
    const int dev = stream_device(st);
    if (dev < 0) return 0;
    int n = cached[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) n = 0;
        cached[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

// Tag of one call's chunk-term flags: a per-process random high half and a call
// counter, never 0 or all ones (what a cleared or 0xFF-filled workspace holds).
// Safe to call from several host threads at once.
uint64_t epoch_salt() {
    static const uint64_t salt = [] {
        static int anchor;
        uint64_t x = (uint64_t)(uintptr_t)&anchor ^ ((uint64_t)time(nullptr) << 20) ^ 0x9e3779b97f4a7c15ull;
        x ^= x >> 33; x *= 0xff51afd7ed558ccdull; x ^= x >> 33;
        return (x & 0x7ffffffeull) + 1;
    }();
    return salt;
}
uint64_t next_epoch() {
    static std::atomic<uint64_t> counter{0};
    return (epoch_salt() << 32) | (uint32_t)(counter.fetch_add(1, std::memory_order_relaxed) + 1);
}

template <typename IO, int DK, bool SNAP = false, bool NORM = false>
void launch_prefill(Params p, long slots, hipStream_t st) {
    if (p.ragged)
        hipLaunchKernelGGL(k_ragged_setup, dim3(1), dim3(NSET), 0, st, p.cu, p.n_seq, p.T, p.seq_start,
                           p.seq_len, p.chunk_off, p.seq_perm, p.cprefix, p.cprefix + (p.cpt + 2), p.cpt, CH);
    if constexpr (sizeof(IO) == 2) {
        // one launch with the chunk terms formed beside the chain when it leaves
        // a quarter of the compute units free; otherwise the chunk terms first
        // (three workgroups per CU) and the chain after, longest sequence first
        const long nchain = (long)p.n_seq * p.H * (p.DV / SL);
        const long items = slots * p.H;
        const long cus = stream_cus(st);
        const long spare = cus - nchain;   // CUs the chain leaves free (one chain workgroup per CU)
        if (spare >= 8 && 4 * spare >= cus && items > 0) {
            p.npw = (int)std::min(spare, (items + 1) / 2);
            p.xcd_items = !p.ragged && p.H % 8 == 0 && p.npw >= 8;
            if (p.xcd_items) p.npw &= ~7;
            p.epoch = next_epoch();
            hipLaunchKernelGGL((k_prefill_fused_bf16<DK, SNAP, NORM>), dim3((unsigned)(p.npw + nchain)), dim3(NT_CHAIN), 0,
                               st, p);
            return;
        }
    }
    if (slots > 0 && p.T > 0) {
        if constexpr (sizeof(IO) == 2)
            hipLaunchKernelGGL((k_chunk_terms_bf16<DK, NORM>), dim3((unsigned)(slots * p.H)), dim3(NT), 0, st, p);
        else
            hipLaunchKernelGGL((k_chunk_terms<DK>), dim3((unsigned)(slots * p.H)), dim3(NT_T32), 0, st, p);
    }
    const dim3 grid((unsigned)(p.n_seq * p.H * (p.DV / SL)));
    if constexpr (sizeof(IO) == 2)
        hipLaunchKernelGGL((k_state_chain_bf16<DK, SNAP, NORM>), grid, dim3(NT_CHAIN), 0, st, p);
    else
        hipLaunchKernelGGL((k_state_chain<DK, SNAP>), grid, dim3(NT_CHAIN), 0, st, p);
}

// ---- evaluation plans: sequential chain, segment-parallel (narrow and wide); workspace; launches
constexpr int SEG_AUTO_MAX = 16;   // most segments per sequence the narrow split chooses by itself
constexpr int SEG_MAX = 64;        // most segments per sequence accepted
constexpr long PLAN_CUS = 256;     // compute units the workspace size assumes
constexpr int PLAN_BITS = GDN_PLAN_SEQUENTIAL | GDN_PLAN_SEGMENTED | GDN_PLAN_WIDE;
enum PlanForm { FORM_AUTO = 0, FORM_SEQ = 1, FORM_SEG = 2, FORM_WIDE = 3 };

struct SegPlan {
    int form = FORM_SEQ;
    int P = 1;   // segments per sequence (1: the sequential form)
    int L = 0;   // chunks per segment
};

int plan_form(int flags) {
    switch (flags & PLAN_BITS) {
        case GDN_PLAN_SEQUENTIAL: return FORM_SEQ;
        case GDN_PLAN_SEGMENTED: return FORM_SEG;
        case GDN_PLAN_WIDE: return FORM_WIDE;
        default: return FORM_AUTO;
    }
}

// Time model of the sequential and narrow segmented forms (microseconds), fitted
// to timings at dk = dv = 128 on a 256-CU MI355X.  The sequential form costs a
// fixed start and one chain step per chunk.  The segmented form costs a fixed
// part (its launches, the chunk terms' start), a part per token and head (chunk
// terms, the output pass), one chain step per chunk of a segment and one scan
// step per segment.  A chain that needs more workgroups than CUs (one per CU:
// its LDS) runs in rounds.
struct SegCost {
    double seq_fixed, chunk, seg_fixed, per_token_head, per_segment;
};
constexpr SegCost COST_BF16 = {17.0, 0.73, 28.5, 3.6e-4, 1.4};
constexpr SegCost COST_F32 = {15.0, 2.0, 30.0, 5.0e-4, 2.0};
// The wide form (dense bf16, 16 segments, every pass one workgroup per
// (sequence, segment, head)): a fixed part (four launches, each pass's first
// loads) and a cost per chunk of a sequence that grows with the units it runs
// beside, from timings at T = 2048..10240 and B H = 1..16.
struct WideCost {
    double fixed, chunk, chunk_per_unit;
};
constexpr WideCost COST_WIDE = {46.0, 0.30, 0.019};

SegPlan split_plan(int form, int nc, int P) {
    SegPlan x;
    P = std::min(P, nc);
    if (P < 2) return x;
    x.L = (nc + P - 1) / P;
    x.P = (nc + x.L - 1) / x.L;   // every segment non-empty
    if (x.P < 2) return SegPlan{};
    x.form = form;
    return x;
}

// The wide form applies to dense bf16 input with dk = dv, without the key
// normalisation transform.
bool wide_applies(int n_seqs, int io, int dk, int dv, int pre) {
    return n_seqs == 0 && io == GDN_BF16 && dk == dv && !(pre & PRE_L2);
}

// Segments of the wide form by itself: about one workgroup per CU in each pass
// (one per (sequence, segment, head)).
int wide_auto_P(int B, int H, int nc) {
    const long units = (long)B * H;
    int P = (int)std::max(2L, std::min(16L, (256 + units - 1) / units));
    return std::min(P, nc);
}

// The plan for a call.  form_req: FORM_* (FORM_AUTO chooses); seg_req: segments
// (0: the form's own count).  Ragged input and snapshots keep the sequential form
// (the caller rejects a forced wide plan that does not apply).
SegPlan choose_plan(int B, int T, int H, int dk, int dv, int n_seqs, int io, int pre, int form_req, int seg_req,
                    long cus) {
    const int nc = (T + CH - 1) / CH;
    if (form_req == FORM_SEQ || seg_req == 1 || n_seqs > 0 || nc < 2) return SegPlan{};
    const bool wide = wide_applies(n_seqs, io, dk, dv, pre);
    if (form_req == FORM_WIDE) return wide ? split_plan(FORM_WIDE, nc, seg_req > 0 ? seg_req : wide_auto_P(B, H, nc))
                                           : SegPlan{};
    if (form_req == FORM_SEG && seg_req > 1) return split_plan(FORM_SEG, nc, seg_req);
    if (cus <= 0) return SegPlan{};
    const SegCost& k = io == GDN_BF16 ? COST_BF16 : COST_F32;
    auto rounds = [&](long wgs) { return (double)((wgs + cus - 1) / cus); };
    const double t_seq = k.seq_fixed + k.chunk * nc * rounds((long)B * H * (dv / SL));
    SegPlan best_plan;
    double best = form_req == FORM_SEG ? 1e300 : 0.9 * t_seq;   // splitting by itself must win by a margin
    for (int P = 2; P <= std::min(SEG_AUTO_MAX, nc); ++P) {
        const SegPlan x = split_plan(FORM_SEG, nc, P);
        if (x.P != P) continue;
        const double t = k.seg_fixed + k.per_token_head * B * H * (double)T +
                         k.chunk * x.L * rounds((long)B * P * H * ((dv + dk) / SL)) + k.per_segment * P;
        if (t < best) { best = t; best_plan = x; }
    }
    if (form_req == FORM_AUTO && wide) {
        const double t = COST_WIDE.fixed + nc * (COST_WIDE.chunk + COST_WIDE.chunk_per_unit * (double)B * H);
        if (t < best) best_plan = split_plan(FORM_WIDE, nc, wide_auto_P(B, H, nc));
    }
    return best_plan;
}

struct SegLayout {
    Layout base;   // ragged layout over the nseq P segments (narrow) or the dense layout (wide)
    size_t S0seg, Iseg, N, M, X, Y, Mlo, total;
};

bool seg_layout(int B, int T, int H, int dk, int dv, int io, const SegPlan& sp, SegLayout* S) {
    const long nseg = (long)B * sp.P;
    if ((long)B * T >= (1L << 31) || nseg >= (1L << 30)) return false;
    const size_t esz = io == GDN_BF16 ? 2 : 4;
    const size_t sv = (size_t)nseg * H * dv * dk * sizeof(float), sk = (size_t)nseg * H * dk * dk * sizeof(float);
    size_t off = 0;
    auto take = [&](size_t bytes) { const size_t at = off; off = round_up(off + bytes, 256); return at; };
    *S = SegLayout{};
    if (sp.form == FORM_WIDE) {
        if (!ws_layout(B, T, H, dk, dv, 0, io, &S->base)) return false;
        off = round_up(S->base.total, 256);
        S->N = take(sv);
        S->M = take(sv / 2);     // high bf16 parts of the identity runs' states
        S->Mlo = take(sv / 2);   // ... and the low parts
        S->X = take(sv);
        S->total = off;
        return true;
    }
    if (!ws_layout(1, B * T, H, dk, dv, (int)nseg, io, &S->base)) return false;
    const size_t tk = (size_t)B * T * H * dk * esz;
    off = round_up(S->base.total, 256);
    S->S0seg = take(sv);
    S->Iseg = take(sk);
    S->N = take(sv);
    S->M = take(sk);
    S->X = take(sv);
    S->Y = take(tk);
    S->total = off;
    return true;
}

// Workspace bytes of a plan (the sequential form's when the plan does not split).
size_t plan_bytes(int B, int T, int H, int dk, int dv, int n_seqs, int io, const SegPlan& sp) {
    if (sp.P > 1) {
        SegLayout S;
        if (seg_layout(B, T, H, dk, dv, io, sp, &S)) return S.total;
    }
    Layout L;
    return ws_layout(B, T, H, dk, dv, n_seqs, io, &L) ? L.total : 0;
}

// The plan a call takes on a device of `cus` CUs: the requested one, with fewer
// segments while the workspace cannot hold it or a grid would overflow, down to
// the sequential form.
SegPlan plan_for_call(int B, int T, int H, int dk, int dv, int n_seqs, int io, int pre, int form_req, int seg_req,
                      size_t workspace_bytes, long cus, SegLayout* S) {
    SegPlan sp = choose_plan(B, T, H, dk, dv, n_seqs, io, pre, form_req, seg_req, cus);
    const long nc = (T + CH - 1) / CH;
    while (sp.P > 1 && !(seg_layout(B, T, H, dk, dv, io, sp, S) && S->total <= workspace_bytes &&
                         (long)B * sp.P * H * ((dv + dk) / SL) < (1L << 31) && (long)B * (nc + SEG_MAX + 8) * H < (1L << 31)))
        sp = split_plan(sp.form, (int)nc, sp.P - 1);
    return sp;
}

template <typename IO, int DK, bool NORM = false>
void launch_segmented(Params p, const SegParams& sq, long slots, hipStream_t st) {
    const long nseg = (long)sq.nseq * sq.P;
    const long per_seg = (long)sq.H * std::max(sq.DV, DK) * DK / 4;   // float4s of one segment's initial states
    hipLaunchKernelGGL((k_segment_prep<DK>), dim3((unsigned)((per_seg + NT - 1) / NT), (unsigned)(nseg + 1)), dim3(NT), 0,
                       st, sq);
    if constexpr (sizeof(IO) == 2)
        hipLaunchKernelGGL((k_chunk_terms_bf16<DK, NORM>), dim3((unsigned)(slots * p.H)), dim3(NT), 0, st, p);
    else
        hipLaunchKernelGGL((k_chunk_terms<DK>), dim3((unsigned)(slots * p.H)), dim3(NT_T32), 0, st, p);
    ChainAlt a;
    a.v = nullptr; a.S0 = sq.Iseg; a.st_t = sizeof(IO) == 2 ? 2 : 1; a.o = const_cast<void*>(sq.Y); a.ST = const_cast<float*>(sq.M); a.DV = DK;
    a.first = (int)(nseg * p.H * (p.DV / SL));
    const dim3 grid((unsigned)(a.first + nseg * p.H * (DK / SL)));
    if constexpr (sizeof(IO) == 2)
        hipLaunchKernelGGL((k_state_chain_pair_bf16<DK, NORM>), grid, dim3(NT_CHAIN), 0, st, p, a);
    else
        hipLaunchKernelGGL((k_state_chain_pair<DK>), grid, dim3(NT_CHAIN), 0, st, p, a);
    const long units = (long)sq.nseq * sq.H;   // (sequence, head) pairs, each on one XCD
    hipLaunchKernelGGL((k_segment_scan<IO, DK>), dim3((unsigned)(8 * ((units + 7) / 8) * (sq.DV / SL))), dim3(DK * 4), 0,
                       st, sq);
    const long cunits = (long)sq.nseq * (sq.P - 1) * sq.H;   // (sequence, segment, head) triples, each on one XCD
    hipLaunchKernelGGL((k_segment_correct<IO, DK>), dim3((unsigned)(8 * ((cunits + 7) / 8) * ((sq.L + 1) / 2))),
                       dim3(NT_CORR), 0, st, sq);
}

// The wide segment-parallel form: chunk terms over all chunks, then the three wide passes.
template <int DK>
void launch_wide(Params p, WideParams w, hipStream_t st) {
    const long BH = (long)w.B * w.H;
    hipLaunchKernelGGL((k_chunk_terms_bf16<DK, false>), dim3((unsigned)(BH * w.NC)), dim3(NT), 0, st, p);
    hipLaunchKernelGGL((k_wide_states<DK>), dim3((unsigned)(BH * (w.P - 1))), dim3(4 * DK), 0, st, w);
    hipLaunchKernelGGL((k_wide_scan<DK>), dim3((unsigned)(8 * ((BH + 7) / 8) * (w.D / 16))), dim3(DK * 4), 0, st, w);
    hipLaunchKernelGGL((k_wide_out<DK>), dim3((unsigned)(BH * w.P)), dim3(4 * DK), 0, st, w);
}

template <typename IO, int DK>
void launch_decode(const void* q, const void* k, const void* v, const float* g, const float* beta,
                   float* S, void* o, int B, int H, int HK, int dv, float scale, int pre, hipStream_t st) {
    const int rows_per_wg = 32;
    dim3 grid((dv + rows_per_wg - 1) / rows_per_wg, B * H);
    hipLaunchKernelGGL((k_decode_step<IO, DK>), grid, dim3(NT), 0, st, (const IO*)q, (const IO*)k,
                       (const IO*)v, g, beta, S, (IO*)o, H, HK, dv, rows_per_wg, scale, pre);
}

template <int DH>
void launch_attention(AttnParams a, hipStream_t st) {
    // Two query tiles per wave (four waves, two per SIMD) halve the LDS reads per
    // product; they pay at d = 128 when the grid gives every CU several workgroups
    // (10k 16-head prompt: 546-554 against 578 us; 2k: 57.6 against 49 us)
    const long wgs = (long)a.nqb * a.B * a.H;
    if constexpr (DH == 128) {
        if (wgs >= 4 * stream_cus(st)) {
            hipLaunchKernelGGL((k_attn_causal<DH, 2>), dim3((unsigned)wgs), dim3(NT_ATT / 2), 0, st, a);
            return;
        }
    }
    hipLaunchKernelGGL((k_attn_causal<DH, 1>), dim3((unsigned)wgs), dim3(NT_ATT), 0, st, a);
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
        case GDN_ERR_WAIT: return "GDN_ERR_WAIT";
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

// Validation shared by the workspace and plan queries; false for arguments the prefill would reject.
static bool sizes_ok(int B, int T, int H, int dk, int dv, int chunk, int n_seqs, int io_dtype, int flags, int segments) {
    if (B < 1 || T < 0 || H < 1 || (chunk != CH && !gen_chunk(chunk)) || n_seqs < 0 || (n_seqs > 0 && B != 1))
        return false;
    if (io_dtype != GDN_F32 && io_dtype != GDN_BF16) return false;
    if ((dk != 64 && dk != 128) || (dv != 64 && dv != 128)) return false;
    if (flags & ~(PRE_L2 | PRE_GATES | PLAN_BITS | GDN_TEST_WITHHOLD)) return false;
    const int pb = flags & PLAN_BITS;
    if (pb & (pb - 1)) return false;   // at most one plan
    if (segments < 0 || segments > SEG_MAX) return false;
    if (segments > 1 && plan_form(flags) != FORM_SEG && plan_form(flags) != FORM_WIDE) return false;
    if (plan_form(flags) == FORM_WIDE && !wide_applies(n_seqs, io_dtype, dk, dv, flags & PRE_L2)) return false;
    Layout L;
    if (chunk != CH)   // the generic path: sequential only
        return (plan_form(flags) == FORM_AUTO || plan_form(flags) == FORM_SEQ) && segments <= 1 &&
               gen_layout(B, T, H, chunk, n_seqs, &L);
    return ws_layout(B, T, H, dk, dv, n_seqs, io_dtype, &L);
}

extern "C" size_t gdn_chunk_prefill_workspace_bytes_ex(int B, int T, int H, int dk, int dv, int chunk, int n_seqs,
                                                       int io_dtype, int flags, int segments) {
    if (!sizes_ok(B, T, H, dk, dv, chunk, n_seqs, io_dtype, flags, segments)) return 0;
    Layout L;
    if (chunk != CH) {
        gen_layout(B, T, H, chunk, n_seqs, &L);
        return L.total;
    }
    ws_layout(B, T, H, dk, dv, n_seqs, io_dtype, &L);
    const SegPlan sp = choose_plan(B, T, H, dk, dv, n_seqs, io_dtype, flags & PRE_L2, plan_form(flags), segments, PLAN_CUS);
    return std::max(L.total, plan_bytes(B, T, H, dk, dv, n_seqs, io_dtype, sp));
}

extern "C" size_t gdn_chunk_prefill_workspace_bytes(int B, int T, int H, int dk, int dv, int chunk,
                                                    int n_seqs, int io_dtype) {
    return gdn_chunk_prefill_workspace_bytes_ex(B, T, H, dk, dv, chunk, n_seqs, io_dtype, 0, 0);
}

extern "C" int gdn_chunk_prefill_plan(int B, int T, int H, int dk, int dv, int n_seqs, int io_dtype, int flags,
                                      int segments, size_t workspace_bytes, void* stream, int* form) {
    if (form) *form = 0;
    if (!sizes_ok(B, T, H, dk, dv, CH, n_seqs, io_dtype, flags, segments)) return 0;
    SegLayout S;
    const SegPlan sp = plan_for_call(B, T, H, dk, dv, n_seqs, io_dtype, flags & PRE_L2, plan_form(flags), segments,
                                     workspace_bytes, stream_cus(reinterpret_cast<hipStream_t>(stream)), &S);
    if (form) *form = sp.P > 1 ? (sp.form == FORM_WIDE ? GDN_PLAN_WIDE : GDN_PLAN_SEGMENTED) : GDN_PLAN_SEQUENTIAL;
    return sp.P;
}

// The prefill behind both entry points: snap_every = 0 takes no snapshots.
static gdn_status prefill(const void* q, const void* k, const void* v, const float* g, const float* beta,
                          const float* S0, void* o, float* S_T, int B, int T, int H, int HK, int dk, int dv, int chunk,
                          const int32_t* cu_seqlens, int n_seqs, int io_dtype, float scale, int flags, int segments,
                          int snap_every, float* snaps, void* workspace, size_t workspace_bytes, void* stream) {
    if (flags & ~(PRE_L2 | PRE_GATES | PLAN_BITS | GDN_TEST_WITHHOLD))
        return fail(GDN_ERR_INVALID_ARG, "flags=%d: unknown bits", flags);
    const int pb = flags & PLAN_BITS, pre = flags & (PRE_L2 | PRE_GATES), form_req = plan_form(flags);
    if (pb & (pb - 1)) return fail(GDN_ERR_INVALID_ARG, "flags=%d: more than one plan", flags);
    if (segments < 0 || segments > SEG_MAX)
        return fail(GDN_ERR_INVALID_ARG, "segments=%d out of range [0, %d]", segments, SEG_MAX);
    if (segments > 1 && form_req != FORM_SEG && form_req != FORM_WIDE)
        return fail(GDN_ERR_INVALID_ARG, "segments=%d needs GDN_PLAN_SEGMENTED or GDN_PLAN_WIDE", segments);
    if (io_dtype != GDN_F32 && io_dtype != GDN_BF16)
        return fail(GDN_ERR_INVALID_ARG, "io_dtype=%d is neither GDN_F32 nor GDN_BF16", io_dtype);
    if (B < 1 || H < 1 || T < 0) return fail(GDN_ERR_INVALID_ARG, "B=%d H=%d T=%d out of range", B, H, T);
    if (HK < 1 || HK > H || H % HK != 0)
        return fail(GDN_ERR_INVALID_ARG, "H_k=%d key heads must divide the H=%d value heads", HK, H);
    gdn_status st = check_dims(dk, dv);
    if (st != GDN_OK) return st;
    if (chunk < 1) return fail(GDN_ERR_INVALID_ARG, "chunk=%d must be positive", chunk);
    if (chunk != CH && !gen_chunk(chunk))
        return fail(GDN_ERR_UNSUPPORTED, "chunk=%d: the chunk length must be 16, 32, 64 or 128", chunk);
    if (chunk != CH && (form_req == FORM_SEG || form_req == FORM_WIDE || segments > 1))
        return fail(GDN_ERR_UNSUPPORTED, "chunk=%d: only the sequential plan (the segmented plans need chunk 64)", chunk);
    if (chunk != CH && snap_every > 0)
        return fail(GDN_ERR_UNSUPPORTED, "chunk=%d: snapshots need chunk 64", chunk);
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
    if ((long)H * (dk > dv ? dk : dv) > (1L << 24))   // 32-bit in-chunk offsets of 64 rows
        return fail(GDN_ERR_UNSUPPORTED, "H=%d too large", H);
    if (form_req == FORM_WIDE && !wide_applies(n_seqs, io_dtype, dk, dv, pre))
        return fail(GDN_ERR_UNSUPPORTED, "GDN_PLAN_WIDE needs dense bf16 input with dk == dv, without GDN_QK_L2NORM");
    if (form_req == FORM_WIDE && snap_every > 0)
        return fail(GDN_ERR_UNSUPPORTED, "GDN_PLAN_WIDE does not take snapshots");
    const int C = chunk;
    Layout L;
    if (!(C == CH ? ws_layout(B, T, H, dk, dv, n_seqs, io_dtype, &L) : gen_layout(B, T, H, C, n_seqs, &L)))
        return fail(GDN_ERR_UNSUPPORTED, "too many chunks x heads for one call");
    if (workspace_bytes < L.total || (L.total > 0 && workspace == nullptr))
        return fail(GDN_ERR_WORKSPACE, "workspace of %zu bytes at %p; %zu bytes needed", workspace_bytes, workspace,
                    L.total);
    if (workspace && !aligned(workspace, 256)) return fail(GDN_ERR_INVALID_ARG, "workspace is not 256-byte aligned");

    Params p;
    p.q = q; p.k = k; p.v = v; p.g = g; p.beta = beta; p.S0 = S0; p.o = o; p.ST = S_T; p.st_t = 0;
    p.B = B; p.T = T; p.H = H; p.DV = dv;
    p.HK = HK; p.G = H / HK;
    p.n_seq = n_seq;
    p.ragged = n_seqs > 0;
    p.NC = (T + C - 1) / C;
    p.C = C;
    p.cu = cu_seqlens;
    char* ws = reinterpret_cast<char*>(workspace);
    p.seq_start = p.ragged ? reinterpret_cast<int32_t*>(ws + L.meta) : nullptr;
    p.seq_len = p.ragged ? p.seq_start + (n_seqs + 1) : nullptr;
    p.chunk_off = p.ragged ? p.seq_len + (n_seqs + 1) : nullptr;
    p.seq_perm = p.ragged ? p.chunk_off + (n_seqs + 1) : nullptr;
    p.cprefix = p.ragged ? p.seq_perm + (n_seqs + 1) : nullptr;
    p.cpt = (T + C - 1) / C;
    p.wsG = reinterpret_cast<float*>(ws + L.G);
    p.wsT = ws + L.T;
    p.wsP = ws + L.P;
    p.wsKQ = ws + L.KQ;
    p.flags = reinterpret_cast<uint64_t*>(ws + L.F);
    p.epoch = 0;
    p.status = reinterpret_cast<uint64_t*>(ws);
    p.wait_bound = (flags & GDN_TEST_WITHHOLD) ? 1 << 10 : 1 << 22;
    p.withhold = (flags & GDN_TEST_WITHHOLD) != 0;
    p.npw = 0;
    p.xcd_items = 0;
    p.scale = scale;
    p.pre = pre;
    p.snaps = snaps;
    p.snap_every = snap_every;
    p.n_snap = snap_every > 0 ? (T - 1) / (snap_every * CH) : 0;
    if (L.total == 0) {
        p.wsG = nullptr; p.wsT = nullptr; p.wsP = nullptr; p.wsKQ = nullptr; p.flags = nullptr; p.status = nullptr;
    }

    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    if (C != CH) {   // chunk lengths other than 64: the generic path (sequential)
        if (io_dtype == GDN_BF16) {
            if (dk == 128) launch_generic<bf16_t, 128>(p, L.slots, hs);
            else launch_generic<bf16_t, 64>(p, L.slots, hs);
        } else {
            if (dk == 128) launch_generic<float, 128>(p, L.slots, hs);
            else launch_generic<float, 64>(p, L.slots, hs);
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return fail(GDN_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
        return GDN_OK;
    }
    // segment-parallel form when the plan splits and the workspace holds it (never
    // with snapshots: the states inside segments are not formed)
    SegLayout S;
    const SegPlan sp = p.n_snap > 0 ? SegPlan{}
                                    : plan_for_call(B, T, H, dk, dv, n_seqs, io_dtype, pre, form_req, segments,
                                                    workspace_bytes, stream_cus(hs), &S);
    if (sp.P > 1 && sp.form == FORM_WIDE) {
        WideParams w;
        w.q = static_cast<const bf16_t*>(q); w.k = static_cast<const bf16_t*>(k); w.v = static_cast<const bf16_t*>(v);
        w.wsG = reinterpret_cast<const float*>(ws + S.base.G);
        w.wsT = reinterpret_cast<const bf16_t*>(ws + S.base.T);
        w.wsP = reinterpret_cast<const bf16_t*>(ws + S.base.P);
        w.o = static_cast<bf16_t*>(o);
        w.S0 = S0;
        w.N = reinterpret_cast<float*>(ws + S.N);
        w.Mhi = reinterpret_cast<bf16_t*>(ws + S.M);
        w.Mlo = reinterpret_cast<bf16_t*>(ws + S.Mlo);
        w.X = reinterpret_cast<float*>(ws + S.X);
        w.ST = S_T;
        w.B = B; w.T = T; w.H = H; w.HK = HK; w.G = H / HK; w.D = dk; w.NC = p.NC; w.P = sp.P; w.L = sp.L;
        w.scale = scale;
        if (dk == 128) launch_wide<128>(p, w, hs);
        else launch_wide<64>(p, w, hs);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return fail(GDN_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
        return GDN_OK;
    }
    if (sp.P > 1) {
        const int nseg = B * sp.P;
        SegParams sq;
        sq.nseq = B; sq.P = sp.P; sq.L = sp.L; sq.T = T; sq.NC = p.NC; sq.H = H; sq.DV = dv; sq.DK = dk;
        sq.S0 = S0;
        sq.S0seg = reinterpret_cast<float*>(ws + S.S0seg);
        sq.Iseg = reinterpret_cast<float*>(ws + S.Iseg);
        sq.N = reinterpret_cast<float*>(ws + S.N);
        sq.M = reinterpret_cast<float*>(ws + S.M);
        sq.X = ws + S.X;
        sq.ST = S_T;
        sq.Y = ws + S.Y;
        sq.o = o;
        // run 1 as a ragged call over the segments
        Params r = p;
        r.B = 1; r.T = B * T; r.n_seq = nseg; r.ragged = 1;
        r.cpt = (r.T + CH - 1) / CH; r.NC = r.cpt;
        r.cu = nullptr;
        r.S0 = sq.S0seg; r.ST = const_cast<float*>(sq.N);
        r.seq_start = reinterpret_cast<int32_t*>(ws + S.base.meta);
        r.seq_len = r.seq_start + (nseg + 1);
        r.chunk_off = r.seq_len + (nseg + 1);
        r.seq_perm = r.chunk_off + (nseg + 1);
        r.cprefix = r.seq_perm + (nseg + 1);   // read only by the one-launch form
        sq.seq_start = r.seq_start; sq.seq_len = r.seq_len; sq.chunk_off = r.chunk_off; sq.seq_perm = r.seq_perm;
        r.wsG = reinterpret_cast<float*>(ws + S.base.G);
        r.wsT = ws + S.base.T;
        r.wsP = ws + S.base.P;
        r.wsKQ = ws + S.base.KQ;
        r.flags = reinterpret_cast<uint64_t*>(ws + S.base.F);
        const bool norm = pre & PRE_L2;
        if (io_dtype == GDN_BF16) {
            if (dk == 128) norm ? launch_segmented<bf16_t, 128, true>(r, sq, S.base.slots, hs)
                                : launch_segmented<bf16_t, 128>(r, sq, S.base.slots, hs);
            else norm ? launch_segmented<bf16_t, 64, true>(r, sq, S.base.slots, hs)
                      : launch_segmented<bf16_t, 64>(r, sq, S.base.slots, hs);
        } else {
            if (dk == 128) launch_segmented<float, 128>(r, sq, S.base.slots, hs);
            else launch_segmented<float, 64>(r, sq, S.base.slots, hs);
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return fail(GDN_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
        return GDN_OK;
    }
    if (p.n_snap > 0) {
        if (io_dtype == GDN_BF16) {
            if (pre & PRE_L2) {
                if (dk == 128) launch_prefill<bf16_t, 128, true, true>(p, L.slots, hs);
                else launch_prefill<bf16_t, 64, true, true>(p, L.slots, hs);
            } else {
                if (dk == 128) launch_prefill<bf16_t, 128, true>(p, L.slots, hs);
                else launch_prefill<bf16_t, 64, true>(p, L.slots, hs);
            }
        } else {
            if (dk == 128) launch_prefill<float, 128, true>(p, L.slots, hs);
            else launch_prefill<float, 64, true>(p, L.slots, hs);
        }
    } else if (io_dtype == GDN_BF16) {
        if (pre & PRE_L2) {
            if (dk == 128) launch_prefill<bf16_t, 128, false, true>(p, L.slots, hs);
            else launch_prefill<bf16_t, 64, false, true>(p, L.slots, hs);
        } else {
            if (dk == 128) launch_prefill<bf16_t, 128>(p, L.slots, hs);
            else launch_prefill<bf16_t, 64>(p, L.slots, hs);
        }
    } else {
        if (dk == 128) launch_prefill<float, 128>(p, L.slots, hs);
        else launch_prefill<float, 64>(p, L.slots, hs);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(GDN_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    return GDN_OK;
}

extern "C" gdn_status gdn_chunk_prefill(const void* q, const void* k, const void* v, const float* g,
                                        const float* beta, const float* S0, void* o, float* S_T, int B,
                                        int T, int H, int dk, int dv, int chunk, const int32_t* cu_seqlens,
                                        int n_seqs, int io_dtype, float scale, void* workspace,
                                        size_t workspace_bytes, void* stream) {
    g_err[0] = '\0';
    return prefill(q, k, v, g, beta, S0, o, S_T, B, T, H, H, dk, dv, chunk, cu_seqlens, n_seqs, io_dtype, scale, 0, 0, 0,
                   nullptr, workspace, workspace_bytes, stream);
}

extern "C" gdn_status gdn_chunk_prefill_grouped(const void* q, const void* k, const void* v, const float* g,
                                                const float* beta, const float* S0, void* o, float* S_T, int B,
                                                int T, int H, int H_k, int dk, int dv, int chunk,
                                                const int32_t* cu_seqlens, int n_seqs, int io_dtype, float scale,
                                                void* workspace, size_t workspace_bytes, void* stream) {
    g_err[0] = '\0';
    return prefill(q, k, v, g, beta, S0, o, S_T, B, T, H, H_k, dk, dv, chunk, cu_seqlens, n_seqs, io_dtype, scale, 0, 0,
                   0, nullptr, workspace, workspace_bytes, stream);
}

extern "C" gdn_status gdn_chunk_prefill_ex(const void* q, const void* k, const void* v, const float* g,
                                           const float* beta, const float* S0, void* o, float* S_T, int B, int T,
                                           int H, int H_k, int dk, int dv, int chunk, const int32_t* cu_seqlens,
                                           int n_seqs, int io_dtype, float scale, int flags, int segments,
                                           void* workspace, size_t workspace_bytes, void* stream) {
    g_err[0] = '\0';
    return prefill(q, k, v, g, beta, S0, o, S_T, B, T, H, H_k, dk, dv, chunk, cu_seqlens, n_seqs, io_dtype, scale, flags,
                   segments, 0, nullptr, workspace, workspace_bytes, stream);
}

// Scratch of gdn_chunk_prefill_noalloc: one copy per device, held by the loaded
// code object until the process ends.  Host code never uses this name as an
// address (on the host it is a stand-in); it uses what noalloc_scratch returns.
static __device__ __align__(256) unsigned char scratch[GDN_NOALLOC_SCRATCH_BYTES];

// Device address of `scratch` on device `dev`, looked up once per device with that
// device current (each device holds its own copy at its own address); nullptr
// when the lookup fails.
static void* noalloc_scratch(int dev) {
    static std::atomic<void*> addr[64];
    if (dev < 0 || dev >= 64) return nullptr;
    void* ptr = addr[dev].load(std::memory_order_acquire);
    if (ptr != nullptr) return ptr;
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    if (cur != dev && hipSetDevice(dev) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || ptr == nullptr) {
        (void)hipGetLastError();
        return nullptr;
    }
    addr[dev].store(ptr, std::memory_order_release);
    return ptr;
}

extern "C" gdn_status gdn_workspace_status(const void* workspace, size_t workspace_bytes, void* stream) {
    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    const void* ws = workspace;
    if (ws == nullptr) {
        const int dev = stream_device(hs);
        ws = dev >= 0 ? noalloc_scratch(dev) : nullptr;
        if (ws == nullptr) return fail(GDN_ERR_HIP, "no device scratch for the stream's device");
    } else if (workspace_bytes < sizeof(uint64_t)) {
        return GDN_OK;
    }
    uint64_t word = 0;
    hipError_t e = hipMemcpyAsync(&word, ws, sizeof(word), hipMemcpyDeviceToHost, hs);
    if (e == hipSuccess) e = hipStreamSynchronize(hs);
    if (e != hipSuccess) return fail(GDN_ERR_HIP, "reading the status word: %s", hipGetErrorString(e));
    if ((word >> 32) != epoch_salt()) return GDN_OK;   // no call of this process gave up here
    e = hipMemsetAsync(const_cast<void*>(ws), 0, sizeof(word), hs);
    if (e == hipSuccess) e = hipStreamSynchronize(hs);
    if (e != hipSuccess) return fail(GDN_ERR_HIP, "clearing the status word: %s", hipGetErrorString(e));
    return fail(GDN_ERR_WAIT, "a chain workgroup of call %u gave up waiting for chunk terms; its outputs are NaN",
                (unsigned)(word & 0xffffffffu));
}

extern "C" gdn_status gdn_chunk_prefill_noalloc(const void* q, const void* k, const void* v, const float* g,
                                                const float* beta, const float* S0, void* o, float* S_T, int B,
                                                int T, int H, int H_k, int dk, int dv, int chunk,
                                                const int32_t* cu_seqlens, int n_seqs, int io_dtype, float scale,
                                                int flags, int segments, void* stream) {
    g_err[0] = '\0';
    // the least any plan needs is the sequential form's workspace; 0 means arguments
    // the prefill rejects, which it then reports itself
    const size_t need = gdn_chunk_prefill_workspace_bytes_ex(B, T, H, dk, dv, chunk, n_seqs, io_dtype,
                                                            GDN_PLAN_SEQUENTIAL, 0);
    if (need > GDN_NOALLOC_SCRATCH_BYTES)
        return fail(GDN_ERR_WORKSPACE, "these sizes need %zu bytes of scratch; gdn_chunk_prefill_noalloc holds %zu",
                    need, (size_t)GDN_NOALLOC_SCRATCH_BYTES);
    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    void* ws = noalloc_scratch(stream_device(hs));
    if (ws == nullptr) return fail(GDN_ERR_HIP, "no device scratch for the stream's device");
    return prefill(q, k, v, g, beta, S0, o, S_T, B, T, H, H_k, dk, dv, chunk, cu_seqlens, n_seqs, io_dtype, scale, flags,
                   segments, 0, nullptr, ws, GDN_NOALLOC_SCRATCH_BYTES, stream);
}

static gdn_status snapshots(const void* q, const void* k, const void* v, const float* g, const float* beta,
                            const float* S0, void* o, float* S_T, int B, int T, int H, int HK, int dk, int dv, int chunk,
                            const int32_t* cu_seqlens, int n_seqs, int io_dtype, float scale, int flags, int snap_every,
                            float* snaps, void* workspace, size_t workspace_bytes, void* stream) {
    if (snap_every < 1) return fail(GDN_ERR_INVALID_ARG, "snap_every=%d must be positive", snap_every);
    if (chunk == CH && T > 0 && (T - 1) / ((long)snap_every * CH) > 0) {
        if (!snaps) return fail(GDN_ERR_INVALID_ARG, "snaps must be non-null when a snapshot falls inside the prompt");
        if (!aligned(snaps, 16)) return fail(GDN_ERR_INVALID_ARG, "snaps %p is not 16-byte aligned", (void*)snaps);
    }
    if ((long)snap_every * CH > (1L << 30)) snap_every = (1 << 30) / CH;   // no snapshot falls inside any prompt
    if (flags & PLAN_BITS) return fail(GDN_ERR_INVALID_ARG, "flags=%d: snapshots take no plan", flags);
    return prefill(q, k, v, g, beta, S0, o, S_T, B, T, H, HK, dk, dv, chunk, cu_seqlens, n_seqs, io_dtype, scale, flags,
                   0, snap_every, snaps, workspace, workspace_bytes, stream);
}

extern "C" gdn_status gdn_chunk_prefill_snapshots(const void* q, const void* k, const void* v, const float* g,
                                                  const float* beta, const float* S0, void* o, float* S_T, int B,
                                                  int T, int H, int dk, int dv, int chunk,
                                                  const int32_t* cu_seqlens, int n_seqs, int io_dtype, float scale,
                                                  int snap_every, float* snaps, void* workspace,
                                                  size_t workspace_bytes, void* stream) {
    g_err[0] = '\0';
    return snapshots(q, k, v, g, beta, S0, o, S_T, B, T, H, H, dk, dv, chunk, cu_seqlens, n_seqs, io_dtype, scale, 0,
                     snap_every, snaps, workspace, workspace_bytes, stream);
}

extern "C" gdn_status gdn_chunk_prefill_snapshots_ex(const void* q, const void* k, const void* v, const float* g,
                                                     const float* beta, const float* S0, void* o, float* S_T, int B,
                                                     int T, int H, int H_k, int dk, int dv, int chunk,
                                                     const int32_t* cu_seqlens, int n_seqs, int io_dtype, float scale,
                                                     int flags, int snap_every, float* snaps, void* workspace,
                                                     size_t workspace_bytes, void* stream) {
    g_err[0] = '\0';
    return snapshots(q, k, v, g, beta, S0, o, S_T, B, T, H, H_k, dk, dv, chunk, cu_seqlens, n_seqs, io_dtype, scale,
                     flags, snap_every, snaps, workspace, workspace_bytes, stream);
}

static gdn_status decode(const void* q, const void* k, const void* v, const float* g, const float* beta, float* S,
                         void* o, int B, int H, int HK, int dk, int dv, int io_dtype, float scale, int pre,
                         void* stream) {
    if (pre & ~(PRE_L2 | PRE_GATES)) return fail(GDN_ERR_INVALID_ARG, "flags=%d: unknown bits", pre);
    if (io_dtype != GDN_F32 && io_dtype != GDN_BF16)
        return fail(GDN_ERR_INVALID_ARG, "io_dtype=%d is neither GDN_F32 nor GDN_BF16", io_dtype);
    if (B < 1 || H < 1) return fail(GDN_ERR_INVALID_ARG, "B=%d H=%d out of range", B, H);
    if (HK < 1 || HK > H || H % HK != 0)
        return fail(GDN_ERR_INVALID_ARG, "H_k=%d key heads must divide the H=%d value heads", HK, H);
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
        if (dk == 128) launch_decode<bf16_t, 128>(q, k, v, g, beta, S, o, B, H, HK, dv, scale, pre, hs);
        else launch_decode<bf16_t, 64>(q, k, v, g, beta, S, o, B, H, HK, dv, scale, pre, hs);
    } else {
        if (dk == 128) launch_decode<float, 128>(q, k, v, g, beta, S, o, B, H, HK, dv, scale, pre, hs);
        else launch_decode<float, 64>(q, k, v, g, beta, S, o, B, H, HK, dv, scale, pre, hs);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(GDN_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    return GDN_OK;
}

extern "C" gdn_status gdn_decode_step(const void* q, const void* k, const void* v, const float* g,
                                      const float* beta, float* S, void* o, int B, int H, int dk, int dv,
                                      int io_dtype, float scale, void* stream) {
    g_err[0] = '\0';
    return decode(q, k, v, g, beta, S, o, B, H, H, dk, dv, io_dtype, scale, 0, stream);
}

extern "C" gdn_status gdn_decode_step_grouped(const void* q, const void* k, const void* v, const float* g,
                                              const float* beta, float* S, void* o, int B, int H, int H_k, int dk,
                                              int dv, int io_dtype, float scale, void* stream) {
    g_err[0] = '\0';
    return decode(q, k, v, g, beta, S, o, B, H, H_k, dk, dv, io_dtype, scale, 0, stream);
}

extern "C" gdn_status gdn_decode_step_ex(const void* q, const void* k, const void* v, const float* g,
                                         const float* beta, float* S, void* o, int B, int H, int H_k, int dk, int dv,
                                         int io_dtype, float scale, int flags, void* stream) {
    g_err[0] = '\0';
    return decode(q, k, v, g, beta, S, o, B, H, H_k, dk, dv, io_dtype, scale, flags, stream);
}

extern "C" gdn_status gdn_attention_prefill(const void* q, const void* k, const void* v, void* o, int B, int T, int H,
                                            int H_kv, int d, const int32_t* cu_seqlens, int n_seqs, int io_dtype,
                                            float scale, void* stream) {
    g_err[0] = '\0';
    if (io_dtype != GDN_F32 && io_dtype != GDN_BF16)
        return fail(GDN_ERR_INVALID_ARG, "io_dtype=%d is neither GDN_F32 nor GDN_BF16", io_dtype);
    if (B < 1 || T < 0 || H < 1) return fail(GDN_ERR_INVALID_ARG, "B=%d T=%d H=%d out of range", B, T, H);
    if (H_kv < 1 || H_kv > H || H % H_kv != 0)
        return fail(GDN_ERR_INVALID_ARG, "H_kv=%d key/value heads must divide the H=%d query heads", H_kv, H);
    if (d < 1) return fail(GDN_ERR_INVALID_ARG, "d=%d must be positive", d);
    if ((cu_seqlens == nullptr) != (n_seqs == 0))
        return fail(GDN_ERR_INVALID_ARG, "cu_seqlens and n_seqs=%d must be given together", n_seqs);
    if (n_seqs < 0) return fail(GDN_ERR_INVALID_ARG, "n_seqs=%d is negative", n_seqs);
    if (n_seqs > 0 && B != 1) return fail(GDN_ERR_INVALID_ARG, "packed sequences need B == 1 (got %d)", B);
    if (cu_seqlens && !aligned(cu_seqlens, 4)) return fail(GDN_ERR_INVALID_ARG, "cu_seqlens is not 4-byte aligned");
    if (d != 64 && d != 128) return fail(GDN_ERR_UNSUPPORTED, "d=%d: only 64 and 128 are implemented", d);
    if (io_dtype != GDN_BF16) return fail(GDN_ERR_UNSUPPORTED, "attention is implemented for bf16 io only");
    if (T > 0 && (!q || !k || !v || !o)) return fail(GDN_ERR_INVALID_ARG, "q, k, v and o must be non-null");
    const void* ptrs[] = {q, k, v, o};
    for (const void* ptr : ptrs)
        if (ptr && !aligned(ptr, 16)) return fail(GDN_ERR_INVALID_ARG, "tensor pointer %p is not 16-byte aligned", ptr);
    if ((long)H * d > (1L << 20)) return fail(GDN_ERR_UNSUPPORTED, "H=%d too large", H);
    // packed: each sequence adds at most one partial block to the dense count
    const long nqb = ((long)T + AQ - 1) / AQ + (n_seqs > 0 ? n_seqs : 0);
    if (nqb * B * H >= (1L << 31)) return fail(GDN_ERR_UNSUPPORTED, "B*T*H too large");
    if (T == 0) return GDN_OK;
    AttnParams a;
    a.q = static_cast<const bf16_t*>(q);
    a.k = static_cast<const bf16_t*>(k);
    a.v = static_cast<const bf16_t*>(v);
    a.o = static_cast<bf16_t*>(o);
    a.B = B; a.T = T; a.H = H; a.HKV = H_kv;
    a.nqb = (int)nqb;
    a.cu = cu_seqlens;
    a.n_seq = n_seqs;
    a.scale_log2 = scale * 1.4426950408889634f;
    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    if (d == 128) launch_attention<128>(a, hs);
    else launch_attention<64>(a, hs);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(GDN_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
    return GDN_OK;
}
