// Chunked prefill for a chunk length C other than 64 (included by gdn.hip, inside its namespace).
//
// Section 3.2 leaves the chunk length free: the chunked form equals the
// token-by-token recurrence at every C.  The kernels tuned for C = 64 build their
// tiles around it; these evaluate the same algebra for C in {16, 32, 128} with
// fp32 arithmetic on the vector units (fp32 fused multiply-adds run at the same
// peak as fp32 MFMA), in three launches:
//   k_gen_gram   per (chunk, head): prefix sums of g in fp64, gamma_r and
//                D_r = exp(G_n - G_r); A = strict_lower(diag(beta) (K K^T o Gamma))
//                and P = lower(Q K^T o Gamma) (C x C, fp32, into the workspace);
//   k_gen_solve  per (chunk, head): T = (I + A)^{-1} blockwise (16 x 16 diagonal
//                blocks by forward substitution, the others one block diagonal at
//                a time); W = diag(D) T diag(beta) and P' = P T diag(beta)
//                overwrite A and P, stored transposed (column-major);
//   k_gen_chain  per (sequence, head, 16 state rows): the inter-chunk recurrence
//                with the outputs,
//                    X = K S^T,  R' = V - diag(gamma) X,  D U = W R',
//                    O = scale (diag(gamma) Q S^T + P' R'),
//                    S^T <- gamma_n S^T + K^T (D U).
// With GDN_QK_L2NORM the rows of q and k are scaled by their reciprocal lengths
// s_q, s_k (kept per token in the workspace); with GDN_GATE_LOGITS g and beta are
// formed from logits where they are read.  Workspace per (chunk slot, head):
// 4 C floats (gamma, D, s_k, s_q), then C x C floats for A / W and for P / P'.
// Every product keeps a small block of outputs per thread in registers and reads
// its operands from LDS as float4 runs.

constexpr int GEN_NT = 256;   // threads per workgroup
constexpr int GEN_RS = 16;    // state rows per chain workgroup

// Tokens [t0, t0 + n) of the chunk in slot `slot`; false for slots past the last chunk.
__device__ __forceinline__ bool gen_item(const Params& p, long slot, long& t0, int& n) {
    const int C = p.C;
    if (p.ragged) {
        if (slot >= tab(p.chunk_off, p.n_seq)) return false;
        int lo = 0, hi = p.n_seq;   // the sequence whose chunk slots hold `slot`
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (tab(p.chunk_off, mid) <= slot) lo = mid; else hi = mid;
        }
        const int c = (int)(slot - tab(p.chunk_off, lo));
        t0 = tab(p.seq_start, lo) + (long)c * C;
        n = min(C, tab(p.seq_len, lo) - c * C);
    } else {
        const int s = (int)(slot / p.NC), c = (int)(slot % p.NC);
        t0 = (long)s * p.T + (long)c * C;
        n = min(C, p.T - c * C);
    }
    return n > 0;
}

__device__ __forceinline__ void gen_gates(const Params& p, long t, int h, float& g, float& b) {
    g = p.g[t * p.H + h];
    b = p.beta[t * p.H + h];
    if (p.pre & PRE_GATES) {
        g = gate_g(g);
        b = gate_beta(b);
    }
}

// Rows [0, R) of width W of an [*, heads, D] io tensor (head hh, first token t0,
// first column col0) into an LDS tile of fp32 with row pitch LDW; rows n.. zero;
// each row times rs[row] when rs is given.  Every 16-byte load is issued before
// the first LDS store, so a tile costs one memory latency.
template <typename IO, int R, int W, int LDW>
__device__ __forceinline__ void gen_stage(float* dst, const IO* src, long t0, int n, int heads, int hh, int D, int col0,
                                          const float* rs = nullptr) {
    constexpr int VE = 16 / sizeof(IO), VPR = W / VE, NV = (R * VPR + GEN_NT - 1) / GEN_NT;
    static_assert(W % VE == 0 && LDW % 4 == 0, "16-byte pieces");
    uint4 buf[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const int i = threadIdx.x + GEN_NT * j, r = i / VPR, cv = i % VPR;
        buf[j] = make_uint4(0, 0, 0, 0);
        if (i < R * VPR && r < n)
            buf[j] = *reinterpret_cast<const uint4*>(src + ((t0 + r) * heads + hh) * (long)D + col0 + cv * VE);
    }
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const int i = threadIdx.x + GEN_NT * j, r = i / VPR, cv = i % VPR;
        if (i < R * VPR) {
            const float m = rs ? rs[r] : 1.f;
            float* d = dst + r * LDW + cv * VE;
            if constexpr (sizeof(IO) == 2) {
                const uint32_t w[4] = {buf[j].x, buf[j].y, buf[j].z, buf[j].w};
                floatx4 lo, hi;
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    lo[2 * e] = __uint_as_float(w[e] << 16) * m;
                    lo[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u) * m;
                    hi[2 * e] = __uint_as_float(w[2 + e] << 16) * m;
                    hi[2 * e + 1] = __uint_as_float(w[2 + e] & 0xffff0000u) * m;
                }
                *reinterpret_cast<floatx4*>(d) = lo;
                *reinterpret_cast<floatx4*>(d + 4) = hi;
            } else {
                *reinterpret_cast<floatx4*>(d) = __builtin_bit_cast(floatx4, buf[j]) * m;
            }
        }
    }
}

// Rows [r0, r0 + R) of a C x C fp32 matrix (rows past C zero) into LDS with row
// pitch LDW, every load first; LDW need not be a multiple of 4.
template <int C, int R, int LDW>
__device__ __forceinline__ void gen_stage_mat(float* dst, const float* src, int r0) {
    constexpr int VPR = C / 4, NV = (R * VPR + GEN_NT - 1) / GEN_NT;
    floatx4 buf[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const int i = threadIdx.x + GEN_NT * j, r = i / VPR, cv = i % VPR;
        buf[j] = floatx4{0.f, 0.f, 0.f, 0.f};
        if (i < R * VPR && r0 + r < C) buf[j] = *reinterpret_cast<const floatx4*>(src + (long)(r0 + r) * C + 4 * cv);
    }
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const int i = threadIdx.x + GEN_NT * j, r = i / VPR, cv = i % VPR;
        if (i < R * VPR)
#pragma unroll
            for (int e = 0; e < 4; ++e) dst[r * LDW + 4 * cv + e] = buf[j][e];
    }
}

__device__ __forceinline__ floatx4 ld4(const float* ptr) { return *reinterpret_cast<const floatx4*>(ptr); }

template <typename IO, int C, int DK>
__global__ __launch_bounds__(GEN_NT) void k_gen_gram(Params p) {
    constexpr int LD = DK + 4, NB = C / 4;
    __shared__ __attribute__((aligned(16))) float sK[C * LD], sQ[C * LD];
    __shared__ double sG[C];
    __shared__ float sB[C], sSk[C], sSq[C];
    const int H = p.H, h = (int)(blockIdx.x % H), tid = threadIdx.x;
    const long slot = blockIdx.x / H;
    long t0;
    int n;
    if (!gen_item(p, slot, t0, n)) return;
    if (tid < C) {
        float gv = 0.f, bv = 0.f;   // rows past the chunk: no decay, no write
        if (tid < n) gen_gates(p, t0 + tid, h, gv, bv);
        sG[tid] = gv;
        sB[tid] = bv;
    }
    const int HK = p.HK, hk = h / p.G;
    gen_stage<IO, C, DK, LD>(sK, static_cast<const IO*>(p.k), t0, n, HK, hk, DK, 0);
    gen_stage<IO, C, DK, LD>(sQ, static_cast<const IO*>(p.q), t0, n, HK, hk, DK, 0);
    __syncthreads();
    if (tid == 0) {   // G_r = g_0 + ... + g_r in fp64 (at most 128 terms)
        double acc = 0.0;
        for (int r = 0; r < C; ++r) {
            acc += sG[r];
            sG[r] = acc;
        }
    }
    if (tid < C) {   // reciprocal row lengths (1 without the transform)
        float a = 0.f, b = 0.f;
        for (int d = 0; d < DK; ++d) {
            a += sK[tid * LD + d] * sK[tid * LD + d];
            b += sQ[tid * LD + d] * sQ[tid * LD + d];
        }
        const bool l2 = p.pre & PRE_L2;
        sSk[tid] = l2 ? (tid < n ? 1.f / sqrtf(a + L2_EPS) : 0.f) : 1.f;
        sSq[tid] = l2 ? (tid < n ? 1.f / sqrtf(b + L2_EPS) : 0.f) : 1.f;
    }
    __syncthreads();
    const long item = slot * H + h;
    float* wg = p.wsG + item * 4 * C;
    if (tid < C) {
        const double G = sG[tid], Gn = sG[n - 1];
        wg[tid] = (float)exp(G);
        wg[C + tid] = tid < n ? (float)exp(Gn - G) : 0.f;
        wg[2 * C + tid] = sSk[tid];
        wg[3 * C + tid] = sSq[tid];
    }
    float* wA = static_cast<float*>(p.wsT) + item * C * C;
    float* wP = static_cast<float*>(p.wsP) + item * C * C;
    // 4 x 4 blocks (rows 4 br.., columns 4 bc..): the lower ones computed, the upper ones zero
    for (int blk = tid; blk < NB * NB; blk += GEN_NT) {
        const int br = blk / NB, bc = blk % NB;
        float kk[4][4] = {}, qk[4][4] = {};
        if (bc <= br && 4 * br < n) {
            for (int d = 0; d < DK; d += 4) {
                floatx4 kr[4], qr[4], kc[4];
#pragma unroll
                for (int a = 0; a < 4; ++a) {
                    kr[a] = ld4(&sK[(4 * br + a) * LD + d]);
                    qr[a] = ld4(&sQ[(4 * br + a) * LD + d]);
                    kc[a] = ld4(&sK[(4 * bc + a) * LD + d]);
                }
#pragma unroll
                for (int a = 0; a < 4; ++a)
#pragma unroll
                    for (int b = 0; b < 4; ++b)
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            kk[a][b] += kr[a][e] * kc[b][e];
                            qk[a][b] += qr[a][e] * kc[b][e];
                        }
            }
        }
#pragma unroll
        for (int a = 0; a < 4; ++a) {
            const int r = 4 * br + a;
            floatx4 av, pv;
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int i = 4 * bc + b;
                av[b] = pv[b] = 0.f;
                if (r < n && i <= r) {
                    const float gam = expf((float)(sG[r] - sG[i]));   // decay masked before it is formed
                    if (i < r) av[b] = sB[r] * gam * kk[a][b] * sSk[r] * sSk[i];
                    pv[b] = gam * qk[a][b] * sSq[r] * sSk[i];
                }
            }
            *reinterpret_cast<floatx4*>(&wA[r * C + 4 * bc]) = av;
            *reinterpret_cast<floatx4*>(&wP[r * C + 4 * bc]) = pv;
        }
    }
}

template <int C>
__global__ __launch_bounds__(GEN_NT) void k_gen_solve(Params p) {
    constexpr int LD = C + 1, NB = C / 16;
    __shared__ float sA[C * LD], sT[C * LD];
    __shared__ float sZ[(NB > 1 ? NB - 1 : 1) * 256];
    __shared__ float sB[C], sD[C];
    const int H = p.H, h = (int)(blockIdx.x % H), tid = threadIdx.x;
    const long slot = blockIdx.x / H;
    long t0;
    int n;
    if (!gen_item(p, slot, t0, n)) return;
    const long item = slot * H + h;
    float* wA = static_cast<float*>(p.wsT) + item * C * C;
    float* wP = static_cast<float*>(p.wsP) + item * C * C;
    gen_stage_mat<C, C, LD>(sA, wA, 0);
    for (int e = tid; e < C * C; e += GEN_NT) sT[(e / C) * LD + e % C] = 0.f;
    if (tid < C) {
        float gv = 0.f, bv = 0.f;
        if (tid < n) gen_gates(p, t0 + tid, h, gv, bv);
        sB[tid] = bv;
        sD[tid] = p.wsG[item * 4 * C + C + tid];
    }
    __syncthreads();
    // diagonal blocks T_bb = (I + A_bb)^{-1}: thread 16 b + j solves column j of block b
    if (tid < C) {
        const int b = tid / 16, j = tid % 16, o = 16 * b;
        float x[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) x[r] = r == j ? 1.f : 0.f;
#pragma unroll
        for (int i = 0; i < 15; ++i)
#pragma unroll
            for (int r = i + 1; r < 16; ++r) x[r] -= sA[(o + r) * LD + o + i] * x[i];
#pragma unroll
        for (int r = 0; r < 16; ++r) sT[(o + r) * LD + o + j] = x[r];
    }
    __syncthreads();
    // block diagonal dd: T_{b,b-dd} = -T_bb Z with Z = sum_{m = b-dd}^{b-1} A_bm T_{m,b-dd}
    for (int dd = 1; dd < NB; ++dd) {
        const int nb = NB - dd;
        for (int e = tid; e < nb * 256; e += GEN_NT) {
            const int b = dd + e / 256, r = (e % 256) / 16, c = e % 16, j = b - dd;
            float acc = 0.f;
            for (int k = 16 * j; k < 16 * b; ++k) acc += sA[(16 * b + r) * LD + k] * sT[k * LD + 16 * j + c];
            sZ[e] = acc;
        }
        __syncthreads();
        for (int e = tid; e < nb * 256; e += GEN_NT) {
            const int b = dd + e / 256, r = (e % 256) / 16, c = e % 16, j = b - dd, zb = e - (e % 256);
            float acc = 0.f;
#pragma unroll
            for (int k = 0; k < 16; ++k) acc += sT[(16 * b + r) * LD + 16 * b + k] * sZ[zb + k * 16 + c];
            sT[(16 * b + r) * LD + 16 * j + c] = -acc;
        }
        __syncthreads();
    }
    // W^T[c][r] = D_r T[r][c] beta_c (column-major W); P into sA
    for (int e = tid; e < C * C; e += GEN_NT) {
        const int c = e / C, r = e % C;
        wA[e] = r < n ? sD[r] * sT[r * LD + c] * sB[c] : 0.f;
    }
    gen_stage_mat<C, C, LD>(sA, wP, 0);
    __syncthreads();
    // P'^T[c][r] = beta_c sum_{c <= i <= r} P[r][i] T[i][c], 4 x 4 blocks of (r, c)
    constexpr int NQ = C / 4;
    for (int blk = tid; blk < NQ * NQ; blk += GEN_NT) {
        const int br = blk % NQ, bc = blk / NQ;
        float acc[4][4] = {};
        if (bc <= br)
            for (int i = 4 * bc; i < 4 * br + 4; ++i) {
                float pr[4], tc[4];
#pragma unroll
                for (int a = 0; a < 4; ++a) {
                    pr[a] = sA[(4 * br + a) * LD + i];
                    tc[a] = sT[i * LD + 4 * bc + a];
                }
#pragma unroll
                for (int a = 0; a < 4; ++a)
#pragma unroll
                    for (int b = 0; b < 4; ++b) acc[a][b] += pr[a] * tc[b];   // T is lower: terms i > r vanish
            }
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int c = 4 * bc + b;
            floatx4 v;
#pragma unroll
            for (int a = 0; a < 4; ++a) v[a] = acc[a][b] * sB[c];
            *reinterpret_cast<floatx4*>(&wP[c * C + 4 * br]) = v;
        }
    }
}

template <typename IO, int C, int DK>
__global__ __launch_bounds__(GEN_NT) void k_gen_chain(Params p) {
    constexpr int LK = DK + 4, RS = GEN_RS, LR = RS + 4;
    constexpr int IB = C < 32 ? C : 32, LW = C + 4;   // rows of W^T and P'^T staged at a time
    __shared__ __attribute__((aligned(16))) float sX[C * LK];   // the chunk's Q rows, then its K rows (times s_k)
    __shared__ __attribute__((aligned(16))) float sS[RS * LK];  // this workgroup's state rows
    __shared__ __attribute__((aligned(16))) float sV[C * LR], sQS[C * LR], sR[C * LR], sU[C * LR];
    __shared__ __attribute__((aligned(16))) float sW[IB * LW], sP[IB * LW];
    __shared__ float sGam[C], sSk[C], sSq[C];
    const int H = p.H, DV = p.DV, tid = threadIdx.x;
    const int per = H * (DV / RS);
    const int s = seq_at_rank(p, blockIdx.x / per);
    const int js = (blockIdx.x % per) / H, h = blockIdx.x % H;
    long start;
    int len, cbase;
    seq_info(p, s, start, len, cbase);
    const long srow0 = ((long)(s * H + h) * DV + js * RS) * DK;
    for (int e = tid; e < RS * DK; e += GEN_NT) sS[(e / DK) * LK + e % DK] = p.S0 ? p.S0[srow0 + e] : 0.f;
    const int HK = p.HK, hk = h / p.G;
    IO* op = static_cast<IO*>(p.o);
    const int nc = (len + C - 1) / C;
    // (tokens 2 tt.., state rows 4 rq..) blocks of the token x row products
    constexpr int NTB = C / 2, NRB = RS / 4;
    // Y[t][r] = sum_d sX[t][d] sS[r][d] for a 2 x 4 block
    auto tokrow = [&](int tt, int rq, float (&y)[2][4]) {
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 4; ++b) y[a][b] = 0.f;
        for (int d = 0; d < DK; d += 4) {
            floatx4 xa[2], sb[4];
#pragma unroll
            for (int a = 0; a < 2; ++a) xa[a] = ld4(&sX[(2 * tt + a) * LK + d]);
#pragma unroll
            for (int b = 0; b < 4; ++b) sb[b] = ld4(&sS[(4 * rq + b) * LK + d]);
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b)
#pragma unroll
                    for (int e = 0; e < 4; ++e) y[a][b] += xa[a][e] * sb[b][e];
        }
    };
    for (int c = 0; c < nc; ++c) {
        const long t0 = start + (long)c * C, item = (long)(cbase + c) * H + h;
        const int n = min(C, len - c * C);
        const float* wg = p.wsG + item * 4 * C;
        const float* WT = static_cast<const float*>(p.wsT) + item * C * C;   // W^T [i][t]
        const float* PT = static_cast<const float*>(p.wsP) + item * C * C;   // P'^T [i][t]
        __syncthreads();   // the previous chunk's reads are done
        gen_stage<IO, C, DK, LK>(sX, static_cast<const IO*>(p.q), t0, n, HK, hk, DK, 0);
        gen_stage<IO, C, RS, LR>(sV, static_cast<const IO*>(p.v), t0, n, H, h, DV, js * RS);
        if (tid < C) {
            sGam[tid] = wg[tid];
            sSk[tid] = wg[2 * C + tid];
            sSq[tid] = wg[3 * C + tid];
        }
        __syncthreads();
        // Q S^T (with the entering state), times gamma s_q
        for (int w = tid; w < NTB * NRB; w += GEN_NT) {
            const int tt = w / NRB, rq = w % NRB;
            if (2 * tt >= n) continue;
            float y[2][4];
            tokrow(tt, rq, y);
#pragma unroll
            for (int a = 0; a < 2; ++a) {
                const int t = 2 * tt + a;
                *reinterpret_cast<floatx4*>(&sQS[t * LR + 4 * rq]) =
                    floatx4{y[a][0], y[a][1], y[a][2], y[a][3]} * (sGam[t] * sSq[t]);
            }
        }
        __syncthreads();
        gen_stage<IO, C, DK, LK>(sX, static_cast<const IO*>(p.k), t0, n, HK, hk, DK, 0, sSk);
        __syncthreads();
        // X = K S^T, R' = V - diag(gamma) X
        for (int w = tid; w < NTB * NRB; w += GEN_NT) {
            const int tt = w / NRB, rq = w % NRB;
            if (2 * tt >= n) continue;
            float y[2][4];
            tokrow(tt, rq, y);
#pragma unroll
            for (int a = 0; a < 2; ++a) {
                const int t = 2 * tt + a;
                *reinterpret_cast<floatx4*>(&sR[t * LR + 4 * rq]) =
                    ld4(&sV[t * LR + 4 * rq]) - sGam[t] * floatx4{y[a][0], y[a][1], y[a][2], y[a][3]};
            }
        }
        // D U = W R' and P' R' over blocks of IB rows of W^T and P'^T staged in LDS, then
        // O = scale (Q S^T diag + P' R'): one block of 4 tokens x 4 rows per thread
        // (C / 4 * RS / 4 <= 256 blocks)
        static_assert((C / 4) * NRB <= GEN_NT, "one output block per thread");
        const int tq = tid / NRB, rq = tid % NRB;
        const bool mine = tid < (C / 4) * NRB && 4 * tq < n;
        float u[4][4] = {}, pr[4][4] = {};
        for (int q0 = 0; q0 < n; q0 += IB) {
            __syncthreads();   // sR complete; the previous block's reads done
            gen_stage_mat<C, IB, LW>(sW, WT, q0);
            gen_stage_mat<C, IB, LW>(sP, PT, q0);
            __syncthreads();
            if (mine)
                for (int i = q0; i < q0 + IB && i < n && i < 4 * tq + 4; ++i) {   // W and P' are lower triangular
                    const floatx4 wv = ld4(&sW[(i - q0) * LW + 4 * tq]), pv = ld4(&sP[(i - q0) * LW + 4 * tq]);
                    const floatx4 rv = ld4(&sR[i * LR + 4 * rq]);
#pragma unroll
                    for (int a = 0; a < 4; ++a)
#pragma unroll
                        for (int b = 0; b < 4; ++b) {
                            u[a][b] += wv[a] * rv[b];
                            pr[a][b] += pv[a] * rv[b];
                        }
                }
        }
        if (mine)
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                const int t = 4 * tq + a;
                *reinterpret_cast<floatx4*>(&sU[t * LR + 4 * rq]) = floatx4{u[a][0], u[a][1], u[a][2], u[a][3]};
                if (t < n) {
                    const floatx4 ov = p.scale * (ld4(&sQS[t * LR + 4 * rq]) + floatx4{pr[a][0], pr[a][1], pr[a][2], pr[a][3]});
                    IO* dst = op + ((t0 + t) * H + h) * (long)DV + js * RS + 4 * rq;
                    if constexpr (sizeof(IO) == 2)
                        *reinterpret_cast<bf16x4*>(dst) = __builtin_convertvector(ov, bf16x4);
                    else
                        *reinterpret_cast<floatx4*>(dst) = ov;
                }
            }
        __syncthreads();
        // S^T <- gamma_n S^T + K^T (D U): blocks of 4 rows x 2 key channels
        const float gn = sGam[n - 1];
        for (int w = tid; w < NRB * (DK / 2); w += GEN_NT) {
            const int rb = w / (DK / 2), d0 = 2 * (w % (DK / 2));
            float a[4][2];
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int e = 0; e < 2; ++e) a[j][e] = gn * sS[(4 * rb + j) * LK + d0 + e];
            for (int t = 0; t < n; ++t) {
                const floatx4 uv = ld4(&sU[t * LR + 4 * rb]);
                const float k0 = sX[t * LK + d0], k1 = sX[t * LK + d0 + 1];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    a[j][0] += k0 * uv[j];
                    a[j][1] += k1 * uv[j];
                }
            }
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int e = 0; e < 2; ++e) sS[(4 * rb + j) * LK + d0 + e] = a[j][e];
        }
    }
    __syncthreads();
    if (p.ST)
        for (int e = tid; e < RS * DK; e += GEN_NT) p.ST[srow0 + e] = sS[(e / DK) * LK + e % DK];
}
