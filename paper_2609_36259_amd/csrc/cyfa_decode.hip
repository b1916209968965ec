// Single-token CyFA decode step in absolute-clock coordinates, in place.
//
// Per (stream, head) (Sec. 3.2, Eqs. cyfa-absolute-recurrence and
// cyfa-absolute-readout):
//   lambda <- lambda + delta                     (Eq. cyfa-cumulative-clock)
//   a = beta U(-lambda) b                        temporal write vector
//   Kbar <- alpha Kbar + a k^T,  o' = Kbar q     (streamed through registers)
//   Vbar <- alpha Vbar + a v^T                   (kept in registers)
//   z = scale M U(lambda) o',  w = softmax(z),  o'' = U(-lambda) M^T w,  M = R Phi
//   o = Vbar^T o''
// The step reads and writes each state once; it is bound by HBM bandwidth.
// Each workgroup issues both of its rows x d float states' loads at its start
// (16-byte loads, consecutive lanes on consecutive addresses), so the value
// state arrives while the key state is updated and the readout runs.  The
// updated states are written back with nontemporal (streaming) stores: nothing
// reads them again within the step, and on this memory system a read-modify-write
// stream with ordinary stores tops out well below one with streaming stores.
#include "cyfa_rows.h"

namespace cyfa {

namespace {

typedef float f32x4_nt __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void store_stream(float4 *p, float4 v) {
    const f32x4_nt t = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(t, reinterpret_cast<f32x4_nt *>(p));
}

// Threads per workgroup: eight waves for 128 storage rows (8 + 8 state float4 and
// 8 readout-matrix rows per thread at d = 128), sixteen for 256 rows.
__host__ __device__ constexpr int dec_threads(int rows) { return rows > kStoreRows ? 1024 : 512; }

template <int DK, int DV, int ROWS, typename Tin>
__global__ __launch_bounds__(dec_threads(ROWS)) void decode_kernel(DecParams p, const float *__restrict__ Mg) {
    constexpr int kThreads = dec_threads(ROWS);
    constexpr int KQ = DK / 4;                       // float4 per key-state row
    constexpr int VQ = DV / 4;                       // float4 per value-state row
    constexpr int KIT = ROWS * KQ / kThreads;        // float4 per thread (key state)
    constexpr int VIT = ROWS * VQ / kThreads;        // float4 per thread (value state)
    constexpr int KROWS_PER_IT = kThreads / KQ;
    constexpr int VROWS_PER_IT = kThreads / VQ;
    constexpr int MQ = ROWS / 4;                     // float4 per readout-matrix row
    constexpr int MIT = ROWS * MQ / kThreads;        // readout-matrix rows per thread
    constexpr int NQ = ROWS / 64;                    // slots per lane in the softmax

    __shared__ float qs[DK], ks[DK], vs[DV];
    __shared__ float a_s[ROWS], op[ROWS], xs[ROWS], ws[ROWS];
    __shared__ float zpart[ROWS][MQ + 1];
    __shared__ float4 ypart[kThreads / MQ][MQ];
    __shared__ float2 cs[ROWS / 2];
    __shared__ float4 opart[kThreads / 64][VQ];

    const int nh = blockIdx.x;
    const int h = nh % p.H;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int m = p.m;
    const int J = (m - 1) / 2;
    const Tin *q = static_cast<const Tin *>(p.q);
    const Tin *k = static_cast<const Tin *>(p.k);
    const Tin *v = static_cast<const Tin *>(p.v);

    // Both state streams are issued first (rows >= m are never touched): the
    // value state arrives while the key state is updated and the readout runs.
    float4 *K4 = reinterpret_cast<float4 *>(p.K + (size_t)nh * ROWS * DK);
    float4 *V4 = reinterpret_cast<float4 *>(p.V + (size_t)nh * ROWS * DV);
    const int ck = tid % KQ, cv = tid % VQ;
    float4 kreg[KIT], vreg[VIT];
#pragma unroll
    for (int it = 0; it < KIT; ++it) {
        const int row = it * KROWS_PER_IT + tid / KQ;
        kreg[it] = row < m ? K4[(size_t)row * KQ + ck] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
        const int row = it * VROWS_PER_IT + tid / VQ;
        vreg[it] = row < m ? V4[(size_t)row * VQ + cv] : make_float4(0.f, 0.f, 0.f, 0.f);
    }

    const float alpha = p.log_alpha ? __expf(p.log_alpha[nh]) : 1.f;
    const float beta = p.beta ? p.beta[nh] : 1.f;
    const double lam = reduce_clock(p.clock[nh] + (double)p.delta[nh], m);

    for (int c = tid; c < DK; c += kThreads) {
        qs[c] = load_as_float(q, (size_t)nh * DK + c);
        ks[c] = load_as_float(k, (size_t)nh * DK + c);
    }
    for (int c = tid; c < DV; c += kThreads) vs[c] = load_as_float(v, (size_t)nh * DV + c);
    if (tid < J) {
        float c, s;
        clock_phase(lam, tid + 1, m, &c, &s);
        cs[tid] = make_float2(c, s);
    }
    __syncthreads();
    if (tid < ROWS) {
        const int i = tid;
        float val = 0.f;
        if (i == 0) {
            val = beta / sqrtf((float)m);
        } else if (i < m) {
            const float2 t = cs[(i - 1) >> 1];
            const float amp = beta * sqrtf(2.0f / (float)m);
            val = (i & 1) ? amp * t.x : -amp * t.y;
        }
        a_s[i] = val;
    }
    __syncthreads();

    // ---- key state: update in place and form o' = Kbar q
    {
        const float4 q4 = make_float4(qs[4 * ck], qs[4 * ck + 1], qs[4 * ck + 2], qs[4 * ck + 3]);
        const float4 k4 = make_float4(ks[4 * ck], ks[4 * ck + 1], ks[4 * ck + 2], ks[4 * ck + 3]);
#pragma unroll
        for (int it = 0; it < KIT; ++it) {
            const int row = it * KROWS_PER_IT + tid / KQ;
            float part = 0.f;
            if (row < m) {
                float4 x = kreg[it];
                const float ar = a_s[row];
                x.x = fmaf(alpha, x.x, ar * k4.x);
                x.y = fmaf(alpha, x.y, ar * k4.y);
                x.z = fmaf(alpha, x.z, ar * k4.z);
                x.w = fmaf(alpha, x.w, ar * k4.w);
                store_stream(&K4[(size_t)row * KQ + ck], x);
                part = x.x * q4.x + x.y * q4.y + x.z * q4.z + x.w * q4.w;
            }
#pragma unroll
            for (int off = 1; off < KQ; off <<= 1) part += __shfl_xor(part, off);
            if (ck == 0) op[row] = row < m ? part : 0.f;
        }
    }
    // ---- value state: update in place, keep the new values for the readout
    {
        const float4 v4 = make_float4(vs[4 * cv], vs[4 * cv + 1], vs[4 * cv + 2], vs[4 * cv + 3]);
#pragma unroll
        for (int it = 0; it < VIT; ++it) {
            const int row = it * VROWS_PER_IT + tid / VQ;
            if (row < m) {
                float4 x = vreg[it];
                const float ar = a_s[row];
                x.x = fmaf(alpha, x.x, ar * v4.x);
                x.y = fmaf(alpha, x.y, ar * v4.y);
                x.z = fmaf(alpha, x.z, ar * v4.z);
                x.w = fmaf(alpha, x.w, ar * v4.w);
                store_stream(&V4[(size_t)row * VQ + cv], x);
                vreg[it] = x;
            }
        }
    }
    __syncthreads();
    // ---- middle step
    if (tid < ROWS) {
        const int i = tid;
        float x = 0.f;
        if (i == 0) {
            x = p.scale * op[0];
        } else if (i < m) {
            const int jj = (i - 1) >> 1;
            const float2 t = cs[jj];
            const float a0 = op[2 * jj + 1], a1 = op[2 * jj + 2];
            x = p.scale * ((i & 1) ? (t.x * a0 - t.y * a1) : (t.y * a0 + t.x * a1));
        }
        xs[i] = x;
    }
    // Thread (column quad cm = tid % 32, row group g = tid / 32) holds rows
    // MIT g .. MIT g + MIT-1, columns 4 cm .. 4 cm + 3 of M (16-byte loads, a
    // wave reading two whole rows per load); the same registers serve z = M x
    // and y = M^T w.
    const int cm = tid % MQ, g = tid / MQ;
    const float4 *M4 = reinterpret_cast<const float4 *>(Mg + (size_t)h * ROWS * ROWS);
    float4 mreg[MIT];
#pragma unroll
    for (int r = 0; r < MIT; ++r) mreg[r] = M4[(size_t)(MIT * g + r) * MQ + cm];
    __syncthreads();
    {
        const float4 x4 = make_float4(xs[4 * cm], xs[4 * cm + 1], xs[4 * cm + 2], xs[4 * cm + 3]);
#pragma unroll
        for (int r = 0; r < MIT; ++r) {
            const float4 mm = mreg[r];
            zpart[MIT * g + r][cm] = mm.x * x4.x + mm.y * x4.y + mm.z * x4.z + mm.w * x4.w;
        }
    }
    __syncthreads();
    if (tid < ROWS) {
        float z = 0.f;
#pragma unroll 8
        for (int c = 0; c < MQ; ++c) z += zpart[tid][c];
        ws[tid] = tid < m ? z : -INFINITY;
    }
    __syncthreads();
    if (wave == 0) {
        float zq[NQ];
        float mx = -INFINITY;
#pragma unroll
        for (int qq = 0; qq < NQ; ++qq) {
            zq[qq] = ws[lane + 64 * qq];
            if (p.logits && lane + 64 * qq < m) p.logits[(size_t)nh * m + lane + 64 * qq] = zq[qq];
            mx = fmaxf(mx, zq[qq]);
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
        float sum = 0.f;
#pragma unroll
        for (int qq = 0; qq < NQ; ++qq) {
            zq[qq] = lane + 64 * qq < m ? __expf(zq[qq] - mx) : 0.f;
            sum += zq[qq];
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
        const float inv = 1.f / sum;
#pragma unroll
        for (int qq = 0; qq < NQ; ++qq) ws[lane + 64 * qq] = zq[qq] * inv;
    }
    __syncthreads();
    {
        // y = M^T w: this thread's rows, then the row groups summed
        float4 y4 = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int r = 0; r < MIT; ++r) {
            const float wr = ws[MIT * g + r];
            y4.x = fmaf(mreg[r].x, wr, y4.x);
            y4.y = fmaf(mreg[r].y, wr, y4.y);
            y4.z = fmaf(mreg[r].z, wr, y4.z);
            y4.w = fmaf(mreg[r].w, wr, y4.w);
        }
        ypart[g][cm] = y4;
    }
    __syncthreads();
    if (tid < ROWS) {
        float y[2] = {0.f, 0.f};
        const int i = tid;
        // the rotation pairs paper columns (2jj+1, 2jj+2); column 0 is DC
        const int c0 = i == 0 ? 0 : (i < m ? 2 * ((i - 1) >> 1) + 1 : 0);
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int c = c0 + e;
            const float *yp4 = reinterpret_cast<const float *>(&ypart[0][0]) + c;
#pragma unroll
            for (int gg = 0; gg < kThreads / MQ; ++gg) y[e] += yp4[gg * MQ * 4];
        }
        float x = 0.f;
        if (i == 0) {
            x = y[0];
        } else if (i < m) {
            const float2 t = cs[(i - 1) >> 1];
            x = (i & 1) ? (t.x * y[0] + t.y * y[1]) : (-t.y * y[0] + t.x * y[1]);
        }
        xs[i] = x;   // o''
    }
    __syncthreads();
    // ---- o = Vbar^T o''
    {
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int it = 0; it < VIT; ++it) {
            const int row = it * VROWS_PER_IT + tid / VQ;
            const float w = xs[row];
            acc.x = fmaf(vreg[it].x, w, acc.x);
            acc.y = fmaf(vreg[it].y, w, acc.y);
            acc.z = fmaf(vreg[it].z, w, acc.z);
            acc.w = fmaf(vreg[it].w, w, acc.w);
        }
        // threads sharing cv within a wave: lanes differing in the bits above log2(VQ)
#pragma unroll
        for (int off = VQ; off < 64; off <<= 1) {
            acc.x += __shfl_xor(acc.x, off);
            acc.y += __shfl_xor(acc.y, off);
            acc.z += __shfl_xor(acc.z, off);
            acc.w += __shfl_xor(acc.w, off);
        }
        if (lane < VQ) opart[wave][cv] = acc;
    }
    __syncthreads();
    if (tid < DV) {
        const int c4 = tid >> 2, comp = tid & 3;
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < kThreads / 64; ++w) {
            const float4 t = opart[w][c4];
            s += comp == 0 ? t.x : comp == 1 ? t.y : comp == 2 ? t.z : t.w;
        }
        store_from_float(static_cast<Tin *>(p.o), (size_t)nh * DV + tid, s);
    }
    if (tid == 0) p.clock[nh] = lam;
}

template <int DK, int DV, int ROWS>
hipError_t launch_rows(const DecParams &p, const float *M, hipStream_t s) {
    const dim3 grid(p.N * p.H), block(dec_threads(ROWS));
    if (p.dtype == 0)
        hipLaunchKernelGGL((decode_kernel<DK, DV, ROWS, float>), grid, block, 0, s, p, M);
    else
        hipLaunchKernelGGL((decode_kernel<DK, DV, ROWS, __hip_bfloat16>), grid, block, 0, s, p, M);
    return hipGetLastError();
}

// 256 storage rows are built for head dims up to 128
template <int DK, int DV>
hipError_t launch_typed(const DecParams &p, const float *M, hipStream_t s) {
    if constexpr (DK <= 128 && DV <= 128) {
        if (p.m > kMaxActive) return launch_rows<DK, DV, kWideRows>(p, M, s);
    }
    return launch_rows<DK, DV, kStoreRows>(p, M, s);
}

template <int DK>
hipError_t launch_dv(const DecParams &p, const float *M, hipStream_t s) {
    if (p.dv == 64) return launch_typed<DK, 64>(p, M, s);
    if (p.dv == 128) return launch_typed<DK, 128>(p, M, s);
    return launch_typed<DK, 256>(p, M, s);
}

}  // namespace

hipError_t launch_decode(const DecParams &p, const float *M, hipStream_t s) {
    if (p.dk == 64) return launch_dv<64>(p, M, s);
    if (p.dk == 128) return launch_dv<128>(p, M, s);
    return launch_dv<256>(p, M, s);
}

}  // namespace cyfa
