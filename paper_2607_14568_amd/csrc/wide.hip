// Wide segment-parallel form of the bf16 prefill (included by gdn.hip, inside its namespace).
//
// The chunk map of section 3.2 is affine in the state, S_{c+1} = S_c M_c + N_c
// (S orientation, dv x dk), so a segment of L chunks composes to
// S_end = S_start M_p + N_p.  Dense input is cut at chunk boundaries into P
// segments per sequence and computed in three passes, every one of them wide:
// a workgroup holds a whole (or half a) state of one head, so the chunk inputs
// it stages in LDS feed 64 or 128 state rows at once instead of 16.
//
//   states (k_wide_states): per (sequence, segment, head) one workgroup runs
//     the segment's chunks twice at once: on the true values from zero -- from
//     S0 for segment 0, whose final state is then the true state entering
//     segment 1 -- giving N_p, and on zero values from the identity, giving M_p
//     (row i of the final state is row i of M_p), kept as high and low bf16 parts;
//   scan (k_wide_scan): X_1 = N_0, X_{p+1} = X_p M_p + N_p, each product as
//     three bf16 products (high x high, high x low, low x high), which keeps
//     the composed states near fp32 precision over all segments;
//   outputs (k_wide_out): per (sequence, segment, head) one workgroup reruns
//     the segment from its entering state X_p with the outputs; the last
//     segment stores S_T.
//
// The chunk terms (W = diag(D) T diag(beta), P' = P T diag(beta), gamma) come
// from the chunk-terms kernel, formed once per (chunk, head) before the passes.
//
// A workgroup is dk / 16 waves, two on each SIMD, so that one wave's products
// overlap the other's operand reads and element-wise work.  A wave keeps 32
// (states pass) or 16 (outputs pass) state rows over all dk key channels as fp32
// MFMA accumulators, so the chunk step needs no exchange between waves:
//     X  = K S^T                      (tokens x rows, contraction over keys)
//     R' = V - diag(gamma) X
//     DU = W R'
//     S^T <- gamma_n S^T + K^T DU
//     O^T = scale (S Q^T diag(gamma) + R'^T P'^T)     (outputs only)
// Each accumulator tile pair packs lane-locally into the next product's operand
// (the contraction orders match the fragment layouts of the chunk terms).  Every
// wave copies its share of chunk c + RING - 1 into an LDS ring while chunk c is
// computed; one LDS barrier per chunk orders the ring.

enum { WIDE_VALUE = 0, WIDE_IDENT = 1, WIDE_OUT = 2 };

struct WideParams {
    const bf16_t* q;
    const bf16_t* k;
    const bf16_t* v;
    const float* wsG;     // chunk terms per (chunk slot, head): gamma_r in the first CH floats
    const bf16_t* wsT;    // W fragments
    const bf16_t* wsP;    // P' fragments
    bf16_t* o;
    const float* S0;      // [B, H, D, D] or null (zero)
    float* N;             // [B, P, H, D, D]: value runs' final states
    bf16_t* Mhi;          // [B, P, H, D, D]: identity runs' final states transposed, in the scan's operand order
    bf16_t* Mlo;          //   ... the part the high bf16 part leaves
    float* X;             // [B, P, H, D, D]: states entering the segments (X_0 = S0)
    float* ST;            // [B, H, D, D] or null
    int B, T, H, HK, G, D, NC, P, L;
    float scale;
};

// LDS of one workgroup: a ring of chunk inputs (K, the values of every state row,
// W and gamma; with outputs also Q and P').
template <int DK, bool OUT> struct WideLds {
    static constexpr int RING = OUT ? 2 : 4;
    bf16_t sK[RING][CH * DK];
    bf16_t sV[RING][CH * DK];
    bf16x8 sW[RING][NFRAG][64];
    float sG[RING][CH];
    bf16_t sQ[OUT ? RING : 1][OUT ? CH * DK : 8];
    bf16x8 sP[OUT ? RING : 1][OUT ? NFRAG : 1][64];
};

// Chunk terms' fragments each wave copies per chunk (NW waves share the six).
template <int NW> constexpr int wide_nwf() { return (NFRAG + NW - 1) / NW; }
// Loads one wave issues per chunk: a compile-time constant, so that the waits on
// the in-order memory counter are exact.
template <int DK, bool OUT> constexpr int wide_loads() {
    constexpr int NW = DK / 16;
    return 2 + 2 + wide_nwf<NW>() + 1 + (OUT ? 2 + wide_nwf<NW>() : 0);   // K, V, W, gamma (Q, P')
}

// One workgroup of NW = DK / 16 waves over the chunks of segment seg of
// sequence b, head h.  States pass: waves [0, NW/2) hold the value run's state
// rows, 32 each, and waves [NW/2, NW) the identity run's (segment 0 has no
// identity run: those waves only copy).  Outputs pass: every wave holds 16 value
// rows.  Every wave also issues its share of the ring's copies.
template <int DK, bool OUT>
__device__ __forceinline__ void wide_body(const WideParams& p, WideLds<DK, OUT>& lds, const int b, const int seg,
                                          const int h) {
    constexpr int NW = DK / 16;
    constexpr int RW = OUT ? 16 : 32;      // state rows per wave
    constexpr int NRT = RW / 16;           // row tiles per wave
    constexpr int RING = WideLds<DK, OUT>::RING;
    constexpr int NKD = DK / 32;           // contraction steps over the key channels
    constexpr int NMD = DK / 16;           // key tiles of the state
    constexpr int NCH = DK / 8;            // 16-byte pieces per K row
    constexpr int RPI = 64 / NCH;          // rows per 1 KB copy
    constexpr int NWF = wide_nwf<NW>();
    constexpr int NI = wide_loads<DK, OUT>();
    static_assert(NCH == 2 * NW, "two K copies per wave");
    const int H = p.H, D = p.D, HK = p.HK, hk = h / p.G;
    const int c0 = seg * p.L, nc = min(p.L, p.NC - c0);
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, lg = lane >> 4;
    const int run = OUT ? WIDE_OUT : (wave < NW / 2 ? WIDE_VALUE : WIDE_IDENT);
    const int rw0 = OUT ? RW * wave : RW * (wave % (NW / 2));   // first state row of this wave
    const bool active = run != WIDE_IDENT || seg > 0;
    auto swz = [](int r) { return ((4 * (r & 3)) | ((r >> 2) & 3)) & (NCH - 1); };
    auto kq = [&](int r, int cc) { return r * DK + (((cc >> 3) ^ swz(r)) << 3) + (cc & 7); };
    auto rows = [&](int c) { return min(CH, p.T - (c0 + c) * CH); };
    auto tok0 = [&](int c) { return (long)b * p.T + (long)(c0 + c) * CH; };
    auto slot = [&](int c) { return ((long)b * p.NC + c0 + c) * H + h; };
    const long mat = (long)D * DK;

    // ---- copies of chunk c into ring slot sl: this wave's K and V row groups
    // (and Q), chunk-term fragments (the six shared out, repeated where there are
    // more waves than fragments) and gamma
    auto issue = [&](int c, int sl) {
        const long t0 = tok0(c);
        const int n = rows(c);
        const uint32_t kbytes = (uint32_t)(((long)(n - 1) * HK + 1) * DK * 2);
        const auto rk = rsrc(p.k + (t0 * HK + hk) * DK, kbytes);
        const auto rq = rsrc(p.q + (t0 * HK + hk) * DK, kbytes);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int i = wave + NW * j, r = RPI * i + lane / NCH;
            const int off = (r * HK * DK + (((lane % NCH) ^ swz(r)) << 3)) * 2;
            bdma16(rk, &lds.sK[sl][RPI * i * DK], off);
            if constexpr (OUT) bdma16(rq, &lds.sQ[sl][RPI * i * DK], off);
        }
        constexpr int PPR = DK / 8, TPL = 64 / PPR;   // 16-byte pieces per token row, tokens per copy
        const auto rv = rsrc(p.v + (t0 * H + h) * D, (uint32_t)(((long)(n - 1) * H * D + D) * 2));
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int i = wave + NW * j;
            bdma16(rv, &lds.sV[sl][i * 512], ((TPL * i + lane / PPR) * H * D + 8 * (lane % PPR)) * 2);
        }
        const long sc = slot(c);
        const auto rw = rsrc(p.wsT + sc * tp_elems<bf16_t>(), tp_elems<bf16_t>() * 2);
        const auto rp = rsrc(p.wsP + sc * tp_elems<bf16_t>(), tp_elems<bf16_t>() * 2);
#pragma unroll
        for (int j = 0; j < NWF; ++j) {
            const int f = (wave + NW * j) % NFRAG;
            bdma16(rw, &lds.sW[sl][f][0], (f * 64 + lane) * 16);
            if constexpr (OUT) bdma16(rp, &lds.sP[sl][f][0], (f * 64 + lane) * 16);
        }
        bdma4(rsrc(p.wsG + sc * GS, GS * 4), &lds.sG[sl][0], lane * 4);
    };

    // ---- initial state: rows rw0 .. rw0 + RW of this wave's run, key channels chan(md) + e
    auto chan = [&](int md) { return 32 * (md >> 1) + 8 * lg + 4 * (md & 1); };
    floatx4 acc[NRT][NMD];
    {
        const float* src = nullptr;
        if (OUT) src = p.X + ((long)(b * p.P + seg) * H + h) * mat;
        else if (run == WIDE_VALUE && seg == 0 && p.S0) src = p.S0 + ((long)b * H + h) * mat;
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) {
            const int row = rw0 + 16 * rt + l16;
#pragma unroll
            for (int md = 0; md < NMD; ++md) {
                if (run == WIDE_IDENT) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[rt][md][e] = chan(md) + e == row ? 1.f : 0.f;
                } else {
                    acc[rt][md] = src ? *reinterpret_cast<const floatx4*>(src + (long)row * DK + chan(md))
                                      : floatx4{0.f, 0.f, 0.f, 0.f};
                }
            }
        }
    }
    // loop-invariant LDS offsets: K^T operands by transpose reads (key tile md,
    // token block kk, half h2) and V values (row tile rt, token tile mt)
    int offT[NMD][2][2], offV[NRT][4];
#pragma unroll
    for (int md = 0; md < NMD; ++md)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2)
                offT[md][kk][h2] = kq(32 * kk + 16 * h2 + 4 * lg + (l16 >> 2), 32 * (md >> 1) + 8 * (l16 & 3) + 4 * (md & 1));
#pragma unroll
    for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) offV[rt][mt] = (16 * mt + 4 * lg + (l16 >> 2)) * DK + rw0 + 16 * rt + 4 * (l16 & 3);

    // ---- one chunk step of this wave's rows on ring slot sl (chunk c).  Each
    // group of products has its LDS reads issued before the products of the
    // group before it, so that their latency hides behind MFMA work.
    auto fence = [] { __builtin_amdgcn_sched_barrier(0); };
    // carried from a chunk's products to its state update: the K^T operands, D U and gamma_n
    bf16x8 ka[NMD][2], db[NRT][2];
    float gn = 0.f;
    auto step = [&](int c, int sl, auto RUN) {
        constexpr int MODE = decltype(RUN)::value;
        const bf16_t* sK = lds.sK[sl];
        const bf16_t* sQ = lds.sQ[OUT ? sl : 0];
        // K (and Q) rows of the token tiles of group g (TG tiles; element j of step kk is key
        // 32 kk + 8 lg + j), two buffers: group g+1's reads go out before group g's products
        constexpr int TG = OUT ? 1 : 2, NG = 4 / TG;
        bf16x8 kf[2][TG][NKD], qf[2][TG][NKD];
        auto read_kq = [&](int g, int buf) {
#pragma unroll
            for (int i = 0; i < TG; ++i)
#pragma unroll
                for (int kk = 0; kk < NKD; ++kk) {
                    const int at = kq(16 * (TG * g + i) + l16, 32 * kk + 8 * lg);
                    kf[buf][i][kk] = *reinterpret_cast<const bf16x8*>(&sK[at]);
                    if constexpr (OUT) qf[buf][i][kk] = *reinterpret_cast<const bf16x8*>(&sQ[at]);
                }
        };
        read_kq(0, 0);
        fence();
        // S_c as bf16 operands
        bf16x8 sb[NRT][NKD];
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
            for (int kk = 0; kk < NKD; ++kk) sb[rt][kk] = pack_bf16(acc[rt][2 * kk], acc[rt][2 * kk + 1]);
        // X = K S^T and (outputs) S Q^T for the token tiles of group g
        floatx4 x[NRT][4], oq[NRT][4];
        auto xprod = [&](int g, int buf) {
#pragma unroll
            for (int i = 0; i < TG; ++i) {
                const int mt = TG * g + i;
#pragma unroll
                for (int rt = 0; rt < NRT; ++rt) {
                    x[rt][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
                    oq[rt][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
                }
#pragma unroll
                for (int kk = 0; kk < NKD; ++kk)
#pragma unroll
                    for (int rt = 0; rt < NRT; ++rt) {
                        x[rt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[buf][i][kk], sb[rt][kk], x[rt][mt], 0, 0, 0);
                        if constexpr (OUT)
                            oq[rt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sb[rt][kk], qf[buf][i][kk], oq[rt][mt], 0, 0, 0);
                    }
            }
        };
        // V values and decays for R'
        short4v vv[NRT][4];
        floatx4 gm[4];
        auto read_vg = [&] {
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                gm[mt] = *reinterpret_cast<const floatx4*>(&lds.sG[sl][16 * mt + 4 * lg]);
                if constexpr (MODE != WIDE_IDENT)
#pragma unroll
                    for (int rt = 0; rt < NRT; ++rt) vv[rt][mt] = lds_tr8(&lds.sV[sl][offV[rt][mt]]);
            }
        };
#pragma unroll
        for (int g = 0; g < NG; ++g) {
            if (g + 1 < NG) read_kq(g + 1, (g + 1) & 1);
            if (g == NG - 1) read_vg();
            fence();
            xprod(g, g & 1);
            fence();
        }
        // W fragments and the first half of the K^T operands of the state update
        bf16x8 wf[NFRAG];
        auto read_kt = [&](int m0) {
#pragma unroll
            for (int md = m0; md < m0 + NMD / 2; ++md)
#pragma unroll
                for (int kk = 0; kk < 2; ++kk) ka[md][kk] = join4(lds_tr8(&sK[offT[md][kk][0]]), lds_tr8(&sK[offT[md][kk][1]]));
        };
#pragma unroll
        for (int f = 0; f < NFRAG; ++f) wf[f] = lds.sW[sl][f][lane];
        read_kt(0);
        fence();
        // R' = V - diag(gamma) X, packed as the operand of W R' (token 32 kk2 + 16 (j/4) + 4 lg + j%4)
        bf16x8 rb[NRT][2];
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) {
            floatx4 r[4];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                if constexpr (MODE == WIDE_IDENT) {
                    r[mt] = -(gm[mt] * x[rt][mt]);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) r[mt][e] = bf(vv[rt][mt][e]) - gm[mt][e] * x[rt][mt][e];
                }
            }
            rb[rt][0] = pack_bf16(r[0], r[1]);
            rb[rt][1] = pack_bf16(r[2], r[3]);
        }
        // D U = W R' (lower triangular: token tile mt takes blocks kk2 <= mt/2)
#pragma unroll
        for (int rt = 0; rt < NRT; ++rt) {
            floatx4 du[4];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                du[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[frag_id(mt, 0)], rb[rt][0], floatx4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                if (mt >= 2) du[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[frag_id(mt, 1)], rb[rt][1], du[mt], 0, 0, 0);
            }
            db[rt][0] = pack_bf16(du[0], du[1]);
            db[rt][1] = pack_bf16(du[2], du[3]);
        }
        if constexpr (OUT) {
            // O^T = scale (S Q^T diag(gamma) + R'^T P'^T): lane holds 4 consecutive rows of token
            // 16 mt + l16; the store's buffer ends at the chunk's last row (stores past it are dropped)
            const auto ro = rsrc(p.o + (tok0(c) * H + h) * D, (uint32_t)(((long)(rows(c) - 1) * H * D + D) * 2));
            typedef int int2v __attribute__((ext_vector_type(2)));
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const float gq = lds.sG[sl][16 * mt + l16];
                const bf16x8 pf0 = lds.sP[sl][frag_id(mt, 0)][lane];
                const bf16x8 pf1 = lds.sP[sl][mt >= 2 ? frag_id(mt, 1) : 0][lane];
#pragma unroll
                for (int rt = 0; rt < NRT; ++rt) {
                    floatx4 op = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rb[rt][0], pf0, floatx4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                    if (mt >= 2) op = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rb[rt][1], pf1, op, 0, 0, 0);
                    const floatx4 ov = p.scale * (gq * oq[rt][mt] + op);
                    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(int2v, __builtin_convertvector(ov, bf16x4)), ro,
                                                          ((16 * mt + l16) * H * D + rw0 + 16 * rt + 4 * lg) * 2, 0, 0);
                }
            }
        }
        fence();
        read_kt(NMD / 2);
        gn = lds.sG[sl][CH - 1];
        fence();
    };
    // S^T <- gamma_n S^T + K^T (D U), from the registers the step left
    auto supdate = [&] {
#pragma unroll
        for (int md = 0; md < NMD; ++md)
#pragma unroll
            for (int rt = 0; rt < NRT; ++rt) {
                acc[rt][md] *= gn;
                acc[rt][md] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[md][0], db[rt][0], acc[rt][md], 0, 0, 0);
                acc[rt][md] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[md][1], db[rt][1], acc[rt][md], 0, 0, 0);
            }
    };

    // ---- the chunk loop: chunks 0 .. RING-2 ahead of the first (past the last
    // chunk the copies repeat it, so every wave's count of loads stays fixed)
    constexpr int NSTORE = OUT ? 4 * NRT : 0;   // output stores a wave issues per chunk
#pragma unroll
    for (int j = 0; j < RING - 1; ++j) issue(min(j, nc - 1), j);
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NI * (RING - 2)) : "memory");
    // Half of the waves run one phase behind: a chunk's state update goes after the
    // next barrier (its operands are in registers, so the ring slot may be refilled),
    // so the two waves sharing a SIMD are in different phases of a chunk (products
    // beside the update, the R' and D U work beside the products) instead of in step.
    const bool rot = wave >= NW / 2;
    for (int c = 0; c < nc; ++c) {
        const int sl = c % RING;
        lds_barrier();   // chunk c resident; chunk c-1's slot free
        issue(min(c + RING - 1, nc - 1), (c + RING - 1) % RING);
        if (rot && c > 0 && active) supdate();   // chunk c-1's
        if (OUT) step(c, sl, Ic<WIDE_OUT>{});
        else if (run == WIDE_VALUE) step(c, sl, Ic<WIDE_VALUE>{});
        else if (active) step(c, sl, Ic<WIDE_IDENT>{});
        if (!rot && active) supdate();
        // chunk c+1's copies landed (this chunk's output stores were issued after them)
        if (active) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NI * (RING - 2) + NSTORE) : "memory");
        else asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NI * (RING - 2)) : "memory");
    }
    if (rot && nc > 0 && active) supdate();
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

    // ---- final states
    if constexpr (OUT) {
        if (p.ST && seg == p.P - 1) {
            float* dst = p.ST + ((long)b * H + h) * mat;
#pragma unroll
            for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
                for (int md = 0; md < NMD; ++md)
                    *reinterpret_cast<floatx4*>(dst + (long)(rw0 + 16 * rt + l16) * DK + chan(md)) = acc[rt][md];
        }
    } else {
        // value run: N_p straight out.  Identity run: M_p transposed, (key channel,
        // identity row), as high and low bf16 parts, through LDS (the ring, free once
        // every wave has passed the barrier) so that the stores are whole 16-byte runs
        static_assert(2 * DK * DK * 2 <= sizeof(lds.sK), "transpose buffer");
        bf16_t* tH = &lds.sK[0][0];
        bf16_t* tL = tH + DK * DK;
        lds_barrier();
        if (run == WIDE_VALUE) {
            float* dst = p.N + ((long)(b * p.P + seg) * H + h) * mat;
#pragma unroll
            for (int rt = 0; rt < NRT; ++rt)
#pragma unroll
                for (int md = 0; md < NMD; ++md)
                    *reinterpret_cast<floatx4*>(dst + (long)(rw0 + 16 * rt + l16) * DK + chan(md)) = acc[rt][md];
        } else if (active) {
#pragma unroll
            for (int rt = 0; rt < NRT; ++rt) {
                const int row = rw0 + 16 * rt + l16;
#pragma unroll
                for (int md = 0; md < NMD; ++md)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float x = acc[rt][md][e];
                        const bf16_t hi = from_f<bf16_t>(x);
                        tH[(chan(md) + e) * DK + row] = hi;
                        tL[(chan(md) + e) * DK + row] = from_f<bf16_t>(x - to_f(hi));
                    }
            }
        }
        lds_barrier();
        if (run == WIDE_IDENT && active) {
            // stored in the scan's operand order: 16-byte piece j of the matrix is lane j % 64 of
            // block j / 64 = (column tile w, contraction block kk); that lane's 8 values are
            // M_p^T[16 w + lane % 16][32 kk + 8 (lane / 16) ..], so every scan load is 1 KB contiguous
            const long base = ((long)(b * p.P + seg) * H + h) * mat;
            for (int j = tid - 64 * (NW / 2); j < DK * DK / 8; j += 64 * (NW / 2)) {
                const int blk = j >> 6, ln = j & 63;
                const int c = 16 * (blk / NKD) + (ln & 15), q = 4 * (blk % NKD) + (ln >> 4);
                const int i = c * (DK / 8) + q;   // piece of the [key channel][identity row] transpose
                *reinterpret_cast<bf16x8*>(p.Mhi + base + 8 * j) = *reinterpret_cast<const bf16x8*>(tH + 8 * i);
                *reinterpret_cast<bf16x8*>(p.Mlo + base + 8 * j) = *reinterpret_cast<const bf16x8*>(tL + 8 * i);
            }
        }
    }
}

// Pass 1: one workgroup per (sequence, segment p < P-1, head), both runs.
template <int DK>
__global__ __launch_bounds__(4 * DK) __attribute__((amdgpu_waves_per_eu(1, 2))) void k_wide_states(WideParams p) {
    __shared__ WideLds<DK, false> lds;
    const int bid = blockIdx.x, H = p.H, P1 = p.P - 1;
    const int h = bid % H, seg = (bid / H) % P1, b = bid / (H * P1);
    wide_body<DK, false>(p, lds, b, seg, h);
}

// Pass 3: one workgroup per (sequence, segment, head).
template <int DK>
__global__ __launch_bounds__(4 * DK) __attribute__((amdgpu_waves_per_eu(1, 2))) void k_wide_out(WideParams p) {
    __shared__ WideLds<DK, true> lds;
    const int bid = blockIdx.x, H = p.H, P = p.P;
    const int h = bid % H, seg = (bid / H) % P, b = bid / (H * P);
    wide_body<DK, true>(p, lds, b, seg, h);
}

// Scan: one workgroup per (sequence, head, 16 state rows); rows never mix.  The
// states X (16 x DK fp32) sit in LDS; wave w forms column tile w of
// X_p M_p + N_p.  A product of an fp32 X and M_p = M_hi + M_lo is taken as
// X_hi M_hi + X_hi M_lo + X_lo M_hi on bf16 MFMA (X_lo = X - X_hi): each term
// rounds at about 2^-16 relative, far below bf16.  M_p arrives transposed and in
// operand order, so a lane's operand is one 16-byte run and a wave's load one
// contiguous kilobyte (lanes reading 16 different rows would touch 16 cache lines
// per load, which runs the load path at a third of its rate).  All 16-row slices of one (sequence, head)
// run on one XCD, whose L2 serves their reads of M_p.
template <int DK>
__global__ __launch_bounds__(DK * 4) void k_wide_scan(WideParams p) {
    constexpr int NTH = DK * 4, NKD = DK / 32;
    __shared__ __attribute__((aligned(16))) float sX[2][16][DK + 4];
    const int H = p.H, P = p.P, nsl = p.D / 16;
    const int xcd = blockIdx.x % 8, k = blockIdx.x / 8;
    const int unit = (k / nsl) * 8 + xcd, js = k % nsl;
    if (unit >= p.B * H) return;
    const int h = unit % H, b = unit / H;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), l16 = lane & 15, lg = lane >> 4;
    const int col = 16 * wave + l16;
    const long mat = (long)p.D * DK;
    auto at = [&](int seg) { return ((long)(b * P + seg) * H + h) * mat; };
    const long rows0 = (long)js * 16 * DK;
    {   // X_0 = S0 (the output pass reads every entering state from X, so S_T may
        // overwrite S0 there), X_1 = N_0 (segment 0's value run started from S0):
        // one float4 of each per thread
        static_assert(16 * DK == 4 * NTH, "one float4 of a 16-row slice per thread");
        const int r = 4 * tid / DK, cc = 4 * tid % DK;
        const floatx4 v = *reinterpret_cast<const floatx4*>(p.N + at(0) + rows0 + 4 * tid);
        const floatx4 s = p.S0 ? *reinterpret_cast<const floatx4*>(p.S0 + ((long)b * H + h) * mat + rows0 + 4 * tid)
                               : floatx4{0.f, 0.f, 0.f, 0.f};
        *reinterpret_cast<floatx4*>(&sX[0][r][cc]) = v;
        *reinterpret_cast<floatx4*>(p.X + at(1) + rows0 + 4 * tid) = v;
        *reinterpret_cast<floatx4*>(p.X + at(0) + rows0 + 4 * tid) = s;
    }
    // M_p and N_p do not depend on X: a ring of R register slots keeps the next R
    // segments' operands in flight, the loop unrolled by R so slots stay fixed
    // (loads never branch: past the last segment they repeat it)
    constexpr int R = 4;
    bf16x8 bh[R][NKD], bl[R][NKD];
    floatx4 nf[R];
    auto load = [&](int seg, auto D) {
        constexpr int d = decltype(D)::value;
        seg = max(1, min(seg, P - 2));
        const bf16_t* mh = p.Mhi + at(seg) + (long)(wave * NKD * 64 + lane) * 8;
        const bf16_t* ml = p.Mlo + at(seg) + (long)(wave * NKD * 64 + lane) * 8;
#pragma unroll
        for (int kk = 0; kk < NKD; ++kk) {
            bh[d][kk] = *reinterpret_cast<const bf16x8*>(mh + kk * 64 * 8);
            bl[d][kk] = *reinterpret_cast<const bf16x8*>(ml + kk * 64 * 8);
        }
        const float* np = p.N + at(seg) + rows0;
#pragma unroll
        for (int e = 0; e < 4; ++e) nf[d][e] = np[(4 * lg + e) * DK + col];
    };
    load(1, Ic<0>{});
    load(2, Ic<1>{});
    load(3, Ic<2>{});
    load(4, Ic<3>{});
    __syncthreads();
    int cur = 0;
    auto step = [&](int seg, auto D) {   // X_{seg+1} = X_seg M_seg + N_seg
        constexpr int d = decltype(D)::value;
        // three independent accumulations (high x high, high x low, low x high), summed at the end
        floatx4 acc = nf[d], a1 = {0.f, 0.f, 0.f, 0.f}, a2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < NKD; ++kk) {
            const floatx4 x0 = *reinterpret_cast<const floatx4*>(&sX[cur][l16][32 * kk + 8 * lg]);
            const floatx4 x1 = *reinterpret_cast<const floatx4*>(&sX[cur][l16][32 * kk + 8 * lg + 4]);
            const bf16x8 xh = pack_bf16(x0, x1);
            floatx4 r0, r1;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                r0[e] = x0[e] - (float)xh[e];
                r1[e] = x1[e] - (float)xh[4 + e];
            }
            const bf16x8 xl = pack_bf16(r0, r1);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xh, bh[d][kk], acc, 0, 0, 0);
            a1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xh, bl[d][kk], a1, 0, 0, 0);
            a2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xl, bh[d][kk], a2, 0, 0, 0);
        }
        acc += a1 + a2;
        load(seg + R, D);
#pragma unroll
        for (int e = 0; e < 4; ++e) sX[cur ^ 1][4 * lg + e][col] = acc[e];
        lds_barrier();
        cur ^= 1;
        {   // X_{seg+1} out as whole 16-byte runs: one float4 per thread
            const int r = 4 * tid / DK, cc = 4 * tid % DK;
            *reinterpret_cast<floatx4*>(p.X + at(seg + 1) + rows0 + 4 * tid) = *reinterpret_cast<const floatx4*>(&sX[cur][r][cc]);
        }
    };
    static_assert(R == 4, "the loop below is unrolled by 4");
    int seg = 1;
    for (; seg + R <= P - 1; seg += R) {
        step(seg, Ic<0>{});
        step(seg + 1, Ic<1>{});
        step(seg + 2, Ic<2>{});
        step(seg + 3, Ic<3>{});
    }
    if (seg < P - 1) step(seg, Ic<0>{});
    if (seg + 1 < P - 1) step(seg + 1, Ic<1>{});
    if (seg + 2 < P - 1) step(seg + 2, Ic<2>{});
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}
