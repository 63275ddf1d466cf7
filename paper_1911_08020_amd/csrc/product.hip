// DARB products for fp32 and fp16 weights (kernels and launch templates in
// product_common.h), and the fused LSTM time step of the recurrent layer.
#include "lstm_cell.h"
#include "product_common.h"

namespace darb {
namespace {

// ---------------------------------------------------------------------------------
// One LSTM time step in one kernel (the recurrent models of section 4.1).  A
// workgroup owns one hidden unit u: its four gate rows u, H+u, 2H+u, 3H+u (in
// different block-size groups, found through the per-row table) are cut into
// chunks of S weights, the workgroup's lane groups take one chunk each, the chunk
// sums meet in LDS in a fixed order and the same workgroup runs the gate cell.
// No data crosses workgroups inside the launch: h_t goes to the other half of a
// double buffer and the next launch reads it.
// ---------------------------------------------------------------------------------

constexpr int kStepThreads = 256;     // 128 / 512 measured slower for 1024 units
constexpr int kMaxStepChunks = 128;
constexpr int kStepBatch = 8;         // gathers in flight per lane (16 measured slower)

template <typename Tw, int CPL, int LGL>
__global__ __launch_bounds__(kStepThreads) void lstm_step_kernel(
    const Tw *__restrict__ values, const uint8_t *__restrict__ offsets,
    const int64_t *__restrict__ rowinfo, int64_t H, int64_t batch,
    const float *__restrict__ h_in, const float *__restrict__ U, int64_t ldu,
    float *__restrict__ c, float *__restrict__ h_out, float *__restrict__ h_seq,
    int64_t ld_seq, int vec_pairs) {
    using XL = XLoad<float, CPL>;
    constexpr int L = 1 << LGL;
    constexpr int GM = L >= 16 ? 1 : 16 / L;
    constexpr int S = L * GM;                           // weights per chunk
    constexpr int NLG = kStepThreads / L;               // lane groups
    constexpr int COLS = L * CPL;                       // batch columns of a lane group
    __shared__ float part[kMaxStepChunks * COLS];

    const int64_t u = blockIdx.x;
    // the unit's gate rows: first slot, block size, chunks (uniform)
    int64_t rs[4];
    int lbs[4], nbs[4], cbeg[5];
    cbeg[0] = 0;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const int64_t info = rowinfo[g * H + u];
        rs[g] = info >> 8;
        lbs[g] = int(info & 0xFF);
        nbs[g] = int((H + (int64_t(1) << lbs[g]) - 1) >> lbs[g]);
        cbeg[g + 1] = cbeg[g] + (nbs[g] + S - 1) / S;
    }
    const int total = cbeg[4];

    // the cell's other inputs, loaded while the products run
    const int tid = int(threadIdx.x);
    float ug[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    float cell_c = 0.0f;
    if (tid < batch) {
#pragma unroll
        for (int g = 0; g < 4; ++g) ug[g] = U[(g * H + u) * ldu + tid];
        cell_c = c[u * batch + tid];
    }

    const int lg = tid / L;
    const int sub = tid & (L - 1);
    const int64_t col0 = int64_t(sub) * CPL;
    const bool col_ok = col0 < batch;
    const int64_t col_c = col_ok ? col0 : 0;
    GroupOffsets go;
    go.u8 = offsets;
    for (int base = 0; base < total; base += NLG) {        // uniform
        const int cid = base + lg;
        const bool cok = cid < total;
        const int cc = cok ? cid : 0;
        const int g = (cc >= cbeg[1] ? 1 : 0) + (cc >= cbeg[2] ? 1 : 0) + (cc >= cbeg[3] ? 1 : 0);
        const int64_t r0 = g == 0 ? rs[0] : g == 1 ? rs[1] : g == 2 ? rs[2] : rs[3];
        const int lb = g == 0 ? lbs[0] : g == 1 ? lbs[1] : g == 2 ? lbs[2] : lbs[3];
        const int nblk = g == 0 ? nbs[0] : g == 1 ? nbs[1] : g == 2 ? nbs[2] : nbs[3];
        const int cb = g == 0 ? cbeg[0] : g == 1 ? cbeg[1] : g == 2 ? cbeg[2] : cbeg[3];
        const int k0 = (cc - cb) * S;                        // < nblk
        const int k = k0 + sub * GM;
        const bool ok = cok && k < nblk;
        float vl[GM];
        int cl[GM];
        {
            float v[GM];
            int o[GM];
            PairLoad<Tw, GM, false>::load(values + r0, go, r0, ok ? k : k0, nblk, vec_pairs != 0,
                                          v, o);
#pragma unroll
            for (int gi = 0; gi < GM; ++gi) {
                const bool okg = ok && k + gi < nblk;
                vl[gi] = okg ? v[gi] : 0.0f;
                const int col = ((k + gi) << lb) + o[gi];
                cl[gi] = okg ? (col < H ? col : int(H) - 1) : -1;   // the encode gives col < H
            }
        }
        float acc[CPL];
#pragma unroll
        for (int q = 0; q < CPL; ++q) acc[q] = 0.0f;
        static_for<0, S / kStepBatch>([&](auto bc) {
            constexpr int b0 = decltype(bc)::value * kStepBatch;
            float vv[kStepBatch];
            int ccl[kStepBatch];
            typename XL::V xv[kStepBatch];
            static_for<0, kStepBatch>([&](auto uc) {
                constexpr int f = b0 + decltype(uc)::value;
                vv[f - b0] = __builtin_bit_cast(
                    float, group_bcast<LGL, f / GM>(__builtin_bit_cast(int, vl[f % GM])));
                ccl[f - b0] = group_bcast<LGL, f / GM>(cl[f % GM]);
                const int64_t x = ccl[f - b0] >= 0 ? ccl[f - b0] : 0;
                xv[f - b0] = XL::load(h_in + x * batch + col_c);
            });
#pragma unroll
            for (int w = 0; w < kStepBatch; ++w) {
                if (ccl[w] >= 0 && col_ok) {
#pragma unroll
                    for (int q = 0; q < CPL; ++q) acc[q] = fmaf(vv[w], XL::get(xv[w], q), acc[q]);
                }
            }
        });
        if (cok) {
#pragma unroll
            for (int q = 0; q < CPL; ++q) part[cid * COLS + sub * CPL + q] = acc[q];
        }
    }
    __syncthreads();
    if (tid < batch) {
        float gate[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            float sum = 0.0f;
            for (int k = cbeg[g]; k < cbeg[g + 1]; ++k) sum += part[k * COLS + tid];
            gate[g] = sum + ug[g];
        }
        float cn = cell_c;
        const float hn = lstm_cell(gate[0], gate[1], gate[2], gate[3], cn);
        c[u * batch + tid] = cn;
        h_out[u * batch + tid] = hn;
        h_seq[u * ld_seq + tid] = hn;
    }
}

// Lanes per gate row for the fused step (batch columns, 4 per lane when aligned), and
// whether the plan's rows fit the chunk table; -1 when the step cannot be fused.
int lstm_step_lgl(const darb_plan &whh, int64_t batch, int cpl) {
    const int64_t lanes = (batch + cpl - 1) / cpl;
    if (lanes > 16) return -1;
    const int lgl = ilog2_ceil(lanes);
    const int64_t S = 16;                               // L * GM for every L <= 16
    int64_t worst = 0;
    for (int g = 0; g < whh.bins.nbins; ++g) {
        const int64_t chunks = (whh.bins.nblk[g] + S - 1) / S;
        if (chunks > worst) worst = chunks;
    }
    return 4 * worst <= kMaxStepChunks ? lgl : -1;
}

template <typename Tw, int CPL>
hipError_t launch_lstm_step_t(const darb_plan &whh, int lgl, const void *values,
                              const uint8_t *offsets, int64_t H, int64_t batch, const float *h_in,
                              const float *U, int64_t ldu, float *c, float *h_out, float *h_seq,
                              int64_t ld_seq, hipStream_t st) {
    const int64_t GM = lgl >= 4 ? 1 : (16 >> lgl);
    bool vec = GM > 1 && reinterpret_cast<uintptr_t>(values) % (GM * sizeof(Tw)) == 0 &&
               reinterpret_cast<uintptr_t>(offsets) % GM == 0;
    for (int g = 0; g < whh.bins.nbins; ++g)
        vec = vec && whh.bins.nblk[g] % GM == 0 && whh.bins.first_elem[g] % GM == 0;
    const Tw *v = static_cast<const Tw *>(values);
#define DARB_STEP(LGL)                                                                          \
    hipLaunchKernelGGL((lstm_step_kernel<Tw, CPL, LGL>), dim3(unsigned(H)), dim3(kStepThreads), \
                       0, st, v, offsets, whh.d_rowinfo, H, batch, h_in, U, ldu, c, h_out,       \
                       h_seq, ld_seq, int(vec))
    switch (lgl) {
        case 0: DARB_STEP(0); break;
        case 1: DARB_STEP(1); break;
        case 2: DARB_STEP(2); break;
        case 3: DARB_STEP(3); break;
        default: DARB_STEP(4); break;
    }
#undef DARB_STEP
    return hipGetLastError();
}

}  // namespace

bool lstm_step_fusable(const darb_plan &whh, int64_t batch, const float *h, const float *h2) {
    const bool vec = batch % 4 == 0 && reinterpret_cast<uintptr_t>(h) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(h2) % 16 == 0;
    return lstm_step_lgl(whh, batch, vec ? 4 : 1) >= 0;
}

hipError_t launch_lstm_step(const darb_plan &whh, int wdtype, const void *values,
                            const uint8_t *offsets, int64_t H, int64_t batch, const float *h_in,
                            const float *U, int64_t ldu, float *c, float *h_out, float *h_seq,
                            int64_t ld_seq, hipStream_t s) {
    // X = h_in and h_out alternate between two buffers; both are aligned alike
    const bool vec = batch % 4 == 0 && reinterpret_cast<uintptr_t>(h_in) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(h_out) % 16 == 0;
    const int lgl = lstm_step_lgl(whh, batch, vec ? 4 : 1);
    if (lgl < 0) return hipErrorInvalidConfiguration;
    if (wdtype == DARB_F32) {
        if (vec) return launch_lstm_step_t<float, 4>(whh, lgl, values, offsets, H, batch, h_in, U,
                                                     ldu, c, h_out, h_seq, ld_seq, s);
        return launch_lstm_step_t<float, 1>(whh, lgl, values, offsets, H, batch, h_in, U, ldu, c,
                                            h_out, h_seq, ld_seq, s);
    }
    if (vec) return launch_lstm_step_t<__half, 4>(whh, lgl, values, offsets, H, batch, h_in, U,
                                                  ldu, c, h_out, h_seq, ld_seq, s);
    return launch_lstm_step_t<__half, 1>(whh, lgl, values, offsets, H, batch, h_in, U, ldu, c,
                                         h_out, h_seq, ld_seq, s);
}

hipError_t launch_spmv(const darb_plan &p, int wdtype, const void *values,
                       const uint8_t *offsets, const uint32_t *packed, int xdtype,
                       const void *x, float *y, hipStream_t s) {
    if (wdtype == DARB_F32)
        return launch_spmv_form<float, float>(p, values, offsets, packed, x, y, nullptr, s);
    if (xdtype == DARB_F16)
        return launch_spmv_form<__half, __half>(p, values, offsets, packed, x, y, nullptr, s);
    return launch_spmv_form<__half, float>(p, values, offsets, packed, x, y, nullptr, s);
}

hipError_t launch_spmm(const darb_plan &p, int wdtype, const void *values,
                       const uint8_t *offsets, const uint32_t *packed, int xdtype, int64_t B,
                       const void *X, int64_t ldx, float *Y, int64_t ldy, hipStream_t s) {
    if (wdtype == DARB_F32)
        return launch_spmm_form<float, float>(p, values, offsets, packed, B, X, ldx, Y, ldy,
                                              nullptr, s);
    if (xdtype == DARB_F16)
        return launch_spmm_form<__half, __half>(p, values, offsets, packed, B, X, ldx, Y, ldy,
                                                nullptr, s);
    return launch_spmm_form<__half, float>(p, values, offsets, packed, B, X, ldx, Y, ldy,
                                           nullptr, s);
}

}  // namespace darb
