// Chunked prefill for a chunk length C other than 64 (included by gdn.hip, inside its namespace).
//
// Section 3.2 leaves the chunk length free: the chunked form equals the
// token-by-token recurrence at every C.  The kernels tuned for C = 64 build their
// tiles around it; these evaluate the same algebra for C in {16, 32, 128} with
// fp32 arithmetic on the vector units, in three launches:
//   k_gen_gram   per (chunk, head): prefix sums of g in fp64, gamma_r and
//                D_r = exp(G_n - G_r); A = strict_lower(diag(beta) (K K^T o Gamma))
//                and P = lower(Q K^T o Gamma) (C x C, fp32, into the workspace);
//   k_gen_solve  per (chunk, head): T = (I + A)^{-1} by forward substitution,
//                one column per thread; W = diag(D) T diag(beta) and
//                P' = P T diag(beta) overwrite A and P;
//   k_gen_chain  per (sequence, head, 16 state rows): the inter-chunk recurrence
//                with the outputs,
//                    X = K S^T,  R' = V - diag(gamma) X,  D U = W R',
//                    O = scale (diag(gamma) Q S^T + P' R'),
//                    S^T <- gamma_n S^T + K^T (D U).
// With GDN_QK_L2NORM the rows of q and k are scaled by their reciprocal lengths
// s_q, s_k (kept per token in the workspace); with GDN_GATE_LOGITS g and beta are
// formed from logits where they are read.  Workspace per (chunk slot, head):
// 4 C floats (gamma, D, s_k, s_q), then C x C floats for A / W and for P / P'.

constexpr int GEN_NT = 256;   // threads per workgroup
constexpr int GEN_RS = 16;    // state rows per chain workgroup

// Tokens [t0, t0 + n) of the chunk in slot `slot`; false for slots past the last chunk.
__device__ __forceinline__ bool gen_item(const Params& p, long slot, long& t0, int& n) {
    const int C = p.C;
    if (p.ragged) {
        if (slot >= p.chunk_off[p.n_seq]) return false;
        int lo = 0, hi = p.n_seq;   // the sequence whose chunk slots hold `slot`
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (p.chunk_off[mid] <= slot) lo = mid; else hi = mid;
        }
        const int c = (int)(slot - p.chunk_off[lo]);
        t0 = p.seq_start[lo] + (long)c * C;
        n = min(C, p.seq_len[lo] - c * C);
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

template <typename IO, int C, int DK>
__global__ __launch_bounds__(GEN_NT) void k_gen_gram(Params p) {
    constexpr int LD = DK + 1;
    __shared__ float sK[C * LD], sQ[C * LD];
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
    const IO* kp = static_cast<const IO*>(p.k);
    const IO* qp = static_cast<const IO*>(p.q);
    for (int i = tid; i < C * DK; i += GEN_NT) {
        const int r = i / DK, d = i % DK;
        float kv = 0.f, qv = 0.f;
        if (r < n) {
            const long at = ((t0 + r) * HK + hk) * (long)DK + d;
            kv = to_f(kp[at]);
            qv = to_f(qp[at]);
        }
        sK[r * LD + d] = kv;
        sQ[r * LD + d] = qv;
    }
    __syncthreads();
    if (tid == 0) {   // G_r = g_0 + ... + g_r in fp64 (a few hundred terms at most)
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
    for (int e = tid; e < C * C; e += GEN_NT) {
        const int r = e / C, i = e % C;
        float a = 0.f, pv = 0.f;
        if (r < n && i <= r) {
            float kk = 0.f, qk = 0.f;
            for (int d = 0; d < DK; ++d) {
                const float ki = sK[i * LD + d];
                kk += sK[r * LD + d] * ki;
                qk += sQ[r * LD + d] * ki;
            }
            const float gam = expf((float)(sG[r] - sG[i]));   // decay masked before it is formed
            if (i < r) a = sB[r] * gam * kk * sSk[r] * sSk[i];
            pv = gam * qk * sSq[r] * sSk[i];
        }
        wA[e] = a;
        wP[e] = pv;
    }
}

template <int C>
__global__ __launch_bounds__(GEN_NT) void k_gen_solve(Params p) {
    constexpr int LD = C + 1;
    __shared__ float sA[C * LD], sT[C * LD];
    __shared__ float sB[C], sD[C];
    const int H = p.H, h = (int)(blockIdx.x % H), tid = threadIdx.x;
    const long slot = blockIdx.x / H;
    long t0;
    int n;
    if (!gen_item(p, slot, t0, n)) return;
    const long item = slot * H + h;
    float* wA = static_cast<float*>(p.wsT) + item * C * C;
    float* wP = static_cast<float*>(p.wsP) + item * C * C;
    for (int e = tid; e < C * C; e += GEN_NT) sA[(e / C) * LD + e % C] = wA[e];
    if (tid < C) {
        float gv = 0.f, bv = 0.f;
        if (tid < n) gen_gates(p, t0 + tid, h, gv, bv);
        sB[tid] = bv;
        sD[tid] = p.wsG[item * 4 * C + C + tid];
    }
    __syncthreads();
    // column j of T = (I + A)^{-1}: T_jj = 1, T_rj = -sum_{j <= i < r} A_ri T_ij
    if (tid < C) {
        const int j = tid;
        for (int r = 0; r < C; ++r) sT[r * LD + j] = r == j ? 1.f : 0.f;
        for (int r = j + 1; r < n; ++r) {
            float acc = 0.f;
            for (int i = j; i < r; ++i) acc += sA[r * LD + i] * sT[i * LD + j];
            sT[r * LD + j] = -acc;
        }
    }
    __syncthreads();
    for (int e = tid; e < C * C; e += GEN_NT) {   // W = diag(D) T diag(beta); P into sA
        const int r = e / C, c = e % C;
        wA[e] = r < n ? sD[r] * sT[r * LD + c] * sB[c] : 0.f;
        sA[r * LD + c] = wP[e];
    }
    __syncthreads();
    for (int e = tid; e < C * C; e += GEN_NT) {   // P' = P T diag(beta) (both lower triangular)
        const int r = e / C, c = e % C;
        float acc = 0.f;
        for (int i = c; i <= r; ++i) acc += sA[r * LD + i] * sT[i * LD + c];
        wP[e] = acc * sB[c];
    }
}

template <typename IO, int C, int DK>
__global__ __launch_bounds__(GEN_NT) void k_gen_chain(Params p) {
    constexpr int LK = DK + 1, RS = GEN_RS, LR = RS + 1;
    __shared__ float sK[C * LK];   // the chunk's key rows (times s_k)
    __shared__ float sS[RS * LK];  // this workgroup's state rows
    __shared__ float sR[C * LR], sU[C * LR];
    __shared__ float sGam[C], sSq[C];
    const int H = p.H, DV = p.DV, tid = threadIdx.x;
    const int per = H * (DV / RS);
    const int s = seq_at_rank(p, blockIdx.x / per);
    const int js = (blockIdx.x % per) / H, h = blockIdx.x % H;
    long start;
    int len, cbase;
    seq_info(p, s, start, len, cbase);
    const long srow0 = ((long)(s * H + h) * DV + js * RS) * DK;
    for (int e = tid; e < RS * DK; e += GEN_NT)
        sS[(e / DK) * LK + e % DK] = p.S0 ? p.S0[srow0 + e] : 0.f;
    const int HK = p.HK, hk = h / p.G;
    const IO* kp = static_cast<const IO*>(p.k);
    const IO* qp = static_cast<const IO*>(p.q);
    const IO* vp = static_cast<const IO*>(p.v);
    IO* op = static_cast<IO*>(p.o);
    const int nc = (len + C - 1) / C;
    for (int c = 0; c < nc; ++c) {
        const long t0 = start + (long)c * C, item = (long)(cbase + c) * H + h;
        const int n = min(C, len - c * C);
        const float* wg = p.wsG + item * 4 * C;
        const float* W = static_cast<const float*>(p.wsT) + item * C * C;
        const float* Pp = static_cast<const float*>(p.wsP) + item * C * C;
        __syncthreads();   // the previous chunk's reads of sK, sR, sU are done
        for (int e = tid; e < C * DK; e += GEN_NT) {
            const int r = e / DK, d = e % DK;
            sK[r * LK + d] = r < n ? to_f(kp[((t0 + r) * HK + hk) * (long)DK + d]) * wg[2 * C + r] : 0.f;
        }
        if (tid < C) {
            sGam[tid] = wg[tid];
            sSq[tid] = wg[3 * C + tid];
        }
        __syncthreads();
        // X = K S^T and R' = V - diag(gamma) X, 4 state rows per work item
        for (int w = tid; w < n * (RS / 4); w += GEN_NT) {
            const int t = w / (RS / 4), r0 = 4 * (w % (RS / 4));
            float x[4] = {0.f, 0.f, 0.f, 0.f};
            for (int d = 0; d < DK; ++d) {
                const float kv = sK[t * LK + d];
#pragma unroll
                for (int j = 0; j < 4; ++j) x[j] += kv * sS[(r0 + j) * LK + d];
            }
#pragma unroll
            for (int j = 0; j < 4; ++j)
                sR[t * LR + r0 + j] = to_f(vp[((t0 + t) * H + h) * (long)DV + js * RS + r0 + j]) - sGam[t] * x[j];
        }
        __syncthreads();
        // D U = W R' and O = scale (diag(gamma) Q S^T + P' R') (S is still the entering state)
        for (int w = tid; w < n * (RS / 4); w += GEN_NT) {
            const int t = w / (RS / 4), r0 = 4 * (w % (RS / 4));
            float u[4] = {0.f, 0.f, 0.f, 0.f}, pr[4] = {0.f, 0.f, 0.f, 0.f}, oq[4] = {0.f, 0.f, 0.f, 0.f};
            for (int i = 0; i <= t; ++i) {
                const float wv = W[t * C + i], pv = Pp[t * C + i];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    u[j] += wv * sR[i * LR + r0 + j];
                    pr[j] += pv * sR[i * LR + r0 + j];
                }
            }
            const IO* qr = qp + ((t0 + t) * HK + hk) * (long)DK;
            for (int d = 0; d < DK; ++d) {
                const float qv = to_f(qr[d]);
#pragma unroll
                for (int j = 0; j < 4; ++j) oq[j] += qv * sS[(r0 + j) * LK + d];
            }
            const float gq = sGam[t] * sSq[t];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                sU[t * LR + r0 + j] = u[j];
                op[((t0 + t) * H + h) * (long)DV + js * RS + r0 + j] = from_f<IO>(p.scale * (gq * oq[j] + pr[j]));
            }
        }
        __syncthreads();
        // S^T <- gamma_n S^T + K^T (D U), 4 state rows per work item
        const float gn = sGam[n - 1];
        for (int w = tid; w < DK * (RS / 4); w += GEN_NT) {
            const int d = w % DK, r0 = 4 * (w / DK);
            float a[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) a[j] = gn * sS[(r0 + j) * LK + d];
            for (int t = 0; t < n; ++t) {
                const float kv = sK[t * LK + d];
#pragma unroll
                for (int j = 0; j < 4; ++j) a[j] += kv * sU[t * LR + r0 + j];
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) sS[(r0 + j) * LK + d] = a[j];
        }
    }
    __syncthreads();
    if (p.ST)
        for (int e = tid; e < RS * DK; e += GEN_NT) p.ST[srow0 + e] = sS[(e / DK) * LK + e % DK];
}
