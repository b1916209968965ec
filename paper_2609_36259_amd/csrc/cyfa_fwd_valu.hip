// Vector-ALU chunk-wise CyFA forward (fp32 arithmetic, any supported shape).
//
// One workgroup per (b, h) sequence walks its chunks in order and keeps both
// absolute-clock states in registers.  Per chunk of C tokens (App. B):
//   clock and log-decay prefix sums      lambda_r (double), G_r = sum log alpha
//   temporal write matrix                A_r = beta_r U(-lambda_r) b  (Eq. app-temporal-writes)
//   key pass     O' = gamma (.) Q Kbar^T + (Q K^T (.) Gamma) A        (Eq. app-cyfa-key-chunk)
//                Kbar <- gamma^C Kbar + (right-rescaled A)^T K
//   middle step  O''_r = U(-lambda_r) M^T softmax(M U(lambda_r) scale O'_r),  M = R Phi
//                                                                   (Eq. cyfa-two-pass, middle line)
//   value pass   O = gamma (.) O'' Vbar + (O'' A^T (.) Gamma) V      (Eq. app-cyfa-value-chunk)
//                Vbar <- gamma^C Vbar + A^T (right-rescaled V)
// gamma^r = exp(G_r), Gamma_rs = exp(G_r - G_s) for r >= s (Eq. app-chunk-decay).
// The basis order inside the kernel is the one of App. A.1 (0 = DC, 2j-1 =
// cos_j, 2j = sin_j); rows m..127 are padding and stay zero.
#include "cyfa_bwd.h"
#include "cyfa_rows.h"

namespace cyfa {

namespace {

constexpr int kValuChunkMax = 16;
// threads per workgroup: 256, or 512 when a head dimension is 256 or the states
// have 256 storage rows (each thread then holds at most 64 + 64 state values;
// with both dimensions at 256 some of the kernel's temporaries spill, which this
// correctness-first fp32 path accepts)
__host__ __device__ constexpr int valu_threads(int dk, int dv, int rows) {
    return (dk > 128 || dv > 128 || rows > kStoreRows) ? 512 : 256;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
    return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

// ROWS: storage rows of the states (128, or 256 for m > 127).  The readout
// matrix sits in LDS with 128 rows and is read from global memory (L2) with 256.
// Chunk groups (gridDim.y > 1): workgroup (b h, g) runs the 16-token chunks
// [g cpg, (g + 1) cpg) starting from the state entering its group (EcK / EcV slot
// g, formed by a pre-pass over the earlier groups' own contributions) and the
// clock entering the group (Eclk slot g, lambda_0 plus the increments before the
// group, from the same pre-pass); the last group writes the final state and
// clock.  No group reads clock0, K0 or V0 itself, so the final state and clock
// may overwrite them in place.  With one group EcK / EcV / Eclk are unused.
template <int DK, int DV, int ROWS, typename Tin>
__global__ __launch_bounds__(valu_threads(DK, DV, ROWS)) void fwd_valu_kernel(FwdParams p, const float *__restrict__ Mg,
                                                                             const float *__restrict__ EcK,
                                                                             const float *__restrict__ EcV,
                                                                             const double *__restrict__ Eclk,
                                                                             int cpg) {
    constexpr int kThreads = valu_threads(DK, DV, ROWS);
    constexpr int CM = kValuChunkMax;
    constexpr int KP = kThreads / ROWS;    // threads sharing a key-state row
    constexpr int KH = DK / KP;            // key-state columns per thread
    constexpr int VP = kThreads / DV;      // threads sharing a value-state column
    constexpr int VR = ROWS / VP;          // value-state rows per thread
    constexpr int MSR = ROWS == kStoreRows ? kStoreRows : 1;   // LDS copy of M (128 rows only)
    constexpr int NJ = ROWS / 2;           // phase-table entries per token

    __shared__ float Qs[CM][DK + 1];
    __shared__ float Ks[CM][DK + 1];
    __shared__ float Vs[CM][DV];
    __shared__ float As[CM][ROWS + 1];
    __shared__ float Ob[CM][ROWS];
    __shared__ float Xb[CM][ROWS];
    __shared__ float Ss[CM][CM];
    __shared__ float Ms[MSR][kStoreRows + 1];
    __shared__ float2 CSs[CM][NJ];
    __shared__ double lam_s[CM];
    __shared__ float G_s[CM];
    __shared__ float beta_s[CM];
    __shared__ double lam_carry;

    const int bh = blockIdx.x, grp = blockIdx.y, G = gridDim.y;
    const int b = bh / p.H, h = bh % p.H;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int m = p.m, C = p.chunk, T = p.T, H = p.H;
    const int Tb = seq_tokens(p, b);                  // this sequence's tokens
    const size_t row0 = seq_row0(p, b);               // its first row
    const int t_lo = G > 1 ? min(grp * cpg * 16, Tb) : 0;
    const int t_hi = G > 1 ? min((grp + 1) * cpg * 16, Tb) : Tb;
    const bool last = grp == G - 1;
    const int J = (m - 1) / 2;
    const float dc = 1.0f / sqrtf((float)m);
    const float ac = sqrtf(2.0f / (float)m);
    const Tin *q = static_cast<const Tin *>(p.q);
    const Tin *k = static_cast<const Tin *>(p.k);
    const Tin *v = static_cast<const Tin *>(p.v);
    Tin *o = static_cast<Tin *>(p.o);

    // state ownership
    const int ki = tid / KP, kh = tid % KP;           // Kbar row ki, columns [kh*KH, kh*KH+KH)
    const int vc = tid / VP, vpart = tid % VP;        // Vbar column vc, rows [vpart*VR, +VR)
    float kst[KH];
    float vst[VR];
    {
        // entering state rows: the initial state [BH][rows][d], or this group's slot of
        // [BH][groups][rows][d]
        const float *K0 = G > 1 ? EcK + ((size_t)bh * G + grp) * ROWS * DK
                                : (p.K0 ? p.K0 + (size_t)bh * ROWS * DK : nullptr);
        const float *V0 = G > 1 ? EcV + ((size_t)bh * G + grp) * ROWS * DV
                                : (p.V0 ? p.V0 + (size_t)bh * ROWS * DV : nullptr);
#pragma unroll
        for (int c = 0; c < KH; ++c) kst[c] = (K0 && ki < m) ? K0[(size_t)ki * DK + kh * KH + c] : 0.f;
#pragma unroll
        for (int ii = 0; ii < VR; ++ii) {
            const int row = vpart * VR + ii;
            vst[ii] = (V0 && row < m) ? V0[(size_t)row * DV + vc] : 0.f;
        }
    }
    const float *Mh = Mg + (size_t)h * ROWS * ROWS;
    if constexpr (ROWS == kStoreRows) {
        for (int e = tid; e < kStoreRows * kStoreRows; e += kThreads)
            Ms[e / kStoreRows][e % kStoreRows] = Mh[e];
    }
    auto Mv = [&](int i, int j) -> float {
        if constexpr (ROWS == kStoreRows) return Ms[i][j];
        else return Mh[i * ROWS + j];
    };
    // clock at the group's first token (with groups: from the pre-pass)
    if (tid == 0) lam_carry = G > 1 ? Eclk[(size_t)bh * G + grp] : reduce_clock(p.clock0 ? p.clock0[bh] : 0.0, m);
    __syncthreads();

    for (int t0 = t_lo; t0 < t_hi; t0 += C) {
        const int n = min(C, t_hi - t0);
        // ---- load the chunk (rows past the end are zero: no write, no decay, no shift)
        for (int e = tid; e < C * DK; e += kThreads) {
            const int r = e / DK, c = e % DK;
            const size_t gi = ((row0 + t0 + r) * H + h) * DK + c;
            Qs[r][c] = r < n ? load_as_float(q, gi) : 0.f;
            Ks[r][c] = r < n ? load_as_float(k, gi) : 0.f;
        }
        for (int e = tid; e < C * DV; e += kThreads) {
            const int r = e / DV, c = e % DV;
            Vs[r][c] = r < n ? load_as_float(v, ((row0 + t0 + r) * H + h) * DV + c) : 0.f;
        }
        if (tid < C) {
            const int r = tid;
            const size_t si = (row0 + t0 + r) * H + h;
            lam_s[r] = r < n ? (double)p.delta[si] : 0.0;
            G_s[r] = (r < n && p.log_alpha) ? p.log_alpha[si] : 0.f;
            beta_s[r] = r < n ? (p.beta ? p.beta[si] : 1.f) : 0.f;
        }
        __syncthreads();
        // ---- clock and log-decay prefix sums (double clock, reduced mod m)
        if (tid == 0) {
            double lam = lam_carry;
            float G = 0.f;
            for (int r = 0; r < C; ++r) {
                lam += lam_s[r];
                lam_s[r] = reduce_clock(lam, m);
                G += G_s[r];
                G_s[r] = G;
            }
            lam_carry = reduce_clock(lam, m);
        }
        __syncthreads();
        for (int e = tid; e < C * J; e += kThreads) {
            const int r = e / J, jj = e % J;
            float c, s;
            clock_phase(lam_s[r], jj + 1, m, &c, &s);
            CSs[r][jj] = make_float2(c, s);
        }
        static_assert(NJ >= kMaxActiveWide / 2 || ROWS == kStoreRows, "phase table holds every pair");
        // S = (Q K^T) (.) Gamma
        for (int e = tid; e < C * C; e += kThreads) {
            const int r = e / C, s = e % C;
            float acc = 0.f;
            if (s <= r) {
                for (int c = 0; c < DK; ++c) acc = fmaf(Qs[r][c], Ks[s][c], acc);
                acc *= __expf(G_s[r] - G_s[s]);
            }
            Ss[r][s] = acc;
        }
        __syncthreads();
        // temporal write matrix A_r = beta_r U(-lambda_r) b
        for (int e = tid; e < C * ROWS; e += kThreads) {
            const int r = e / ROWS, i = e % ROWS;
            const float be = beta_s[r];
            float val = 0.f;
            if (i == 0) {
                val = be * dc;
            } else if (i < m) {
                const float2 cs = CSs[r][(i - 1) >> 1];
                val = (i & 1) ? be * ac * cs.x : -be * ac * cs.y;
            }
            As[r][i] = val;
        }
        // key pass, inter-chunk part: O'_r = gamma^r Kbar q_r (old state)
        for (int r = 0; r < C; ++r) {
            float part = 0.f;
#pragma unroll
            for (int c = 0; c < KH; ++c) part = fmaf(Qs[r][kh * KH + c], kst[c], part);
#pragma unroll
            for (int off = 1; off < KP; off <<= 1) part += __shfl_xor(part, off);
            if (kh == 0) Ob[r][ki] = __expf(G_s[r]) * part;
        }
        __syncthreads();
        // key pass, intra-chunk part: O' += S A
        for (int e = tid; e < C * ROWS; e += kThreads) {
            const int r = e / ROWS, i = e % ROWS;
            float acc = Ob[r][i];
            for (int s = 0; s <= r; ++s) acc = fmaf(Ss[r][s], As[s][i], acc);
            Ob[r][i] = acc;
        }
        // key state carry: Kbar <- gamma^C Kbar + (right-rescaled A)^T K
        {
            const float Glast = G_s[C - 1];
            const float gC = __expf(Glast);
#pragma unroll
            for (int c = 0; c < KH; ++c) kst[c] *= gC;
            for (int r = 0; r < C; ++r) {
                const float w = As[r][ki] * __expf(Glast - G_s[r]);
#pragma unroll
                for (int c = 0; c < KH; ++c) kst[c] = fmaf(w, Ks[r][kh * KH + c], kst[c]);
            }
        }
        __syncthreads();
        // middle step: X_r = U(lambda_r) (scale O'_r)
        for (int e = tid; e < C * ROWS; e += kThreads) {
            const int r = e / ROWS, i = e % ROWS;
            float x = 0.f;
            if (i == 0) {
                x = p.scale * Ob[r][0];
            } else if (i < m) {
                const int jj = (i - 1) >> 1;
                const float2 cs = CSs[r][jj];
                const float a0 = Ob[r][2 * jj + 1], a1 = Ob[r][2 * jj + 2];
                x = p.scale * ((i & 1) ? (cs.x * a0 - cs.y * a1) : (cs.y * a0 + cs.x * a1));
            }
            Xb[r][i] = x;
        }
        __syncthreads();
        // slot logits Z_r = M X_r
        for (int e = tid; e < C * ROWS; e += kThreads) {
            const int r = e / ROWS, i = e % ROWS;
            float acc = 0.f;
            if (i < m) {
                for (int j = 0; j < m; ++j) acc = fmaf(Mv(i, j), Xb[r][j], acc);
                if (p.logits && r < n)
                    p.logits[((row0 + t0 + r) * H + h) * m + i] = acc;
            }
            Ob[r][i] = acc;
        }
        __syncthreads();
        // softmax over the m active slots (padding slots excluded)
        for (int r = wave; r < C; r += kThreads / 64) {
            constexpr int NQ = ROWS / 64;
            float z[NQ];
            float mx = -INFINITY;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                z[q] = lane + 64 * q < m ? Ob[r][lane + 64 * q] : -INFINITY;
                mx = fmaxf(mx, z[q]);
            }
            mx = wave_max(mx);
            float sum = 0.f;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                z[q] = lane + 64 * q < m ? __expf(z[q] - mx) : 0.f;
                sum += z[q];
            }
            const float inv = 1.f / wave_sum(sum);
#pragma unroll
            for (int q = 0; q < NQ; ++q) Ob[r][lane + 64 * q] = z[q] * inv;
        }
        __syncthreads();
        // Y_r = M^T W_r
        for (int e = tid; e < C * ROWS; e += kThreads) {
            const int r = e / ROWS, j = e % ROWS;
            float acc = 0.f;
            if (j < m)
                for (int i = 0; i < m; ++i) acc = fmaf(Ob[r][i], Mv(i, j), acc);
            Xb[r][j] = acc;
        }
        __syncthreads();
        // O''_r = U(-lambda_r) Y_r
        for (int e = tid; e < C * ROWS; e += kThreads) {
            const int r = e / ROWS, i = e % ROWS;
            float x = 0.f;
            if (i == 0) {
                x = Xb[r][0];
            } else if (i < m) {
                const int jj = (i - 1) >> 1;
                const float2 cs = CSs[r][jj];
                const float a0 = Xb[r][2 * jj + 1], a1 = Xb[r][2 * jj + 2];
                x = (i & 1) ? (cs.x * a0 + cs.y * a1) : (-cs.y * a0 + cs.x * a1);
            }
            Ob[r][i] = x;
        }
        __syncthreads();
        // value pass: S2 = (O'' A^T) (.) Gamma
        for (int e = tid; e < C * C; e += kThreads) {
            const int r = e / C, s = e % C;
            float acc = 0.f;
            if (s <= r) {
                for (int i = 0; i < m; ++i) acc = fmaf(Ob[r][i], As[s][i], acc);
                acc *= __expf(G_s[r] - G_s[s]);
            }
            Ss[r][s] = acc;
        }
        __syncthreads();
        // O_r = gamma^r Vbar^T O''_r + sum_s S2_rs V_s
        for (int r = 0; r < C; ++r) {
            float part = 0.f;
#pragma unroll
            for (int ii = 0; ii < VR; ++ii) part = fmaf(Ob[r][vpart * VR + ii], vst[ii], part);
#pragma unroll
            for (int off = 1; off < VP; off <<= 1) part += __shfl_xor(part, off);
            if (vpart == 0 && r < n) {
                float acc = __expf(G_s[r]) * part;
                for (int s = 0; s <= r; ++s) acc = fmaf(Ss[r][s], Vs[s][vc], acc);
                store_from_float(o, ((row0 + t0 + r) * H + h) * DV + vc, acc);
            }
        }
        // value state carry: Vbar <- gamma^C Vbar + A^T (right-rescaled V)
        {
            const float Glast = G_s[C - 1];
            const float gC = __expf(Glast);
#pragma unroll
            for (int ii = 0; ii < VR; ++ii) vst[ii] *= gC;
            for (int r = 0; r < C; ++r) {
                const float w = Vs[r][vc] * __expf(Glast - G_s[r]);
#pragma unroll
                for (int ii = 0; ii < VR; ++ii) vst[ii] = fmaf(As[r][vpart * VR + ii], w, vst[ii]);
            }
        }
        __syncthreads();
    }

    if (p.K_out && last) {
        const size_t kbase = ((size_t)bh * ROWS + ki) * DK + kh * KH;
#pragma unroll
        for (int c = 0; c < KH; ++c) p.K_out[kbase + c] = ki < m ? kst[c] : 0.f;
    }
    if (p.V_out && last) {
#pragma unroll
        for (int ii = 0; ii < VR; ++ii) {
            const int row = vpart * VR + ii;
            p.V_out[((size_t)bh * ROWS + row) * DV + vc] = row < m ? vst[ii] : 0.f;
        }
    }
    if (p.clock_out && last && tid == 0) p.clock_out[bh] = lam_carry;
}

template <int DK, int DV, int ROWS>
hipError_t launch_rows(const FwdParams &p, const float *M, const float *EcK, const float *EcV, const double *Eclk,
                       int groups, int cpg, hipStream_t s) {
    const dim3 grid(p.B * p.H, groups), block(valu_threads(DK, DV, ROWS));
    if (p.dtype == 0)
        hipLaunchKernelGGL((fwd_valu_kernel<DK, DV, ROWS, float>), grid, block, 0, s, p, M, EcK, EcV, Eclk, cpg);
    else
        hipLaunchKernelGGL((fwd_valu_kernel<DK, DV, ROWS, __hip_bfloat16>), grid, block, 0, s, p, M, EcK, EcV, Eclk, cpg);
    return hipGetLastError();
}

// 256 storage rows are built for head dims up to 128
template <int DK, int DV>
hipError_t launch_typed(const FwdParams &p, const float *M, const float *EcK, const float *EcV, const double *Eclk,
                        int groups, int cpg, hipStream_t s) {
    if constexpr (DK <= 128 && DV <= 128) {
        if (p.m > kMaxActive) return launch_rows<DK, DV, kWideRows>(p, M, EcK, EcV, Eclk, groups, cpg, s);
    }
    return launch_rows<DK, DV, kStoreRows>(p, M, EcK, EcV, Eclk, groups, cpg, s);
}

}  // namespace

int valu_chunk_max() { return kValuChunkMax; }

template <int DK>
hipError_t launch_dv(const FwdParams &p, const float *M, const float *EcK, const float *EcV, const double *Eclk,
                     int groups, int cpg, hipStream_t s) {
    if (p.dv == 64) return launch_typed<DK, 64>(p, M, EcK, EcV, Eclk, groups, cpg, s);
    if (p.dv == 128) return launch_typed<DK, 128>(p, M, EcK, EcV, Eclk, groups, cpg, s);
    return launch_typed<DK, 256>(p, M, EcK, EcV, Eclk, groups, cpg, s);
}

bool valu_groups_supported(const FwdParams &p) {
    return p.dk <= 128 && p.dv <= 128 && p.m <= kMaxActive;
}

int valu_auto_groups(const FwdParams &p) {
    if (!valu_groups_supported(p)) return 1;
    const int nc16 = (p.T + 15) / 16;
    const int BH = p.B * p.H;
    int g = (512 + BH - 1) / BH;
    if (g > nc16) g = nc16;
    return g < 1 ? 1 : g;
}

size_t valu_group_workspace_bytes(const FwdParams &p, int groups) {
    return groups > 1 ? group_states_bytes(p.B, p.H, p.dk, p.dv, groups) : 0;
}

// groups > 1: chunk groups of cpg 16-token chunks, their entering states formed in ws
hipError_t launch_fwd_valu(const FwdParams &p, const float *M, int groups, void *ws, hipStream_t s) {
    const float *EcK = nullptr, *EcV = nullptr;
    const double *Eclk = nullptr;
    const int nc16 = (p.T + 15) / 16;
    int cpg = 1;
    if (groups > 1) {
        cpg = (nc16 + groups - 1) / groups;
        groups = (nc16 + cpg - 1) / cpg;
    }
    if (groups > 1) {
        hipError_t e = launch_group_states(p, groups, cpg, ws, &EcK, &EcV, &Eclk, s);
        if (e != hipSuccess) return e;
    } else {
        groups = 1;
    }
    if (p.dk == 64) return launch_dv<64>(p, M, EcK, EcV, Eclk, groups, cpg, s);
    if (p.dk == 128) return launch_dv<128>(p, M, EcK, EcV, Eclk, groups, cpg, s);
    return launch_dv<256>(p, M, EcK, EcV, Eclk, groups, cpg, s);
}

}  // namespace cyfa
