// Decode regime of the gated delta rule (paper: appendix "Operator Background
// and Mathematical Definitions", subsection "Gated Delta Net"): one new token
// per sequence, state updated in place.
//
// Per (b, h) with alpha = exp(g), using the regrouping
//     S alpha (I - beta k k^T) + beta v k^T = alpha S + u k^T,
//     u = beta (v - alpha S k),
// each state row i needs two dot products with the OLD row, kv_i = S_i . k and
// sq_i = S_i . q, after which
//     S'_i = alpha S_i + u_i k^T,
//     o_i  = scale * S'_i . q = scale * (alpha sq_i + u_i (k . q)).
// So every state row is independent given (k, q, alpha, beta, v_i): the kernel
// streams each fp32 state row from HBM once, reduces the two dots across the
// lanes that hold the row, updates it in registers and writes it back.
//
// Layout in a wave: a row of D fp32 is held by LPR = min(8, D/4) consecutive
// lanes, each owning J = D / (4 LPR) float4 column slots at float4 index
// j * LPR + c (c = lane % LPR).  For D = 128 a group of 8 lanes covers one
// 512-byte row with four fully used 128-byte segments, 8 rows per wave
// instruction, RS row sets per wave.  A workgroup of W waves covers
// W * RS * (64 / LPR) consecutive rows of one head; the host picks W so that
// small batches still launch enough workgroups to fill the chip.  State loads
// and stores are non-temporal: every state is touched once per step.
#include "gdn_device.h"
#include "gdn_launch.h"

namespace gdn {

// INDEXED: the state of batch entry b is pool slot idx[b] (entries outside
// [0, P) are skipped) instead of state b.
template <int D, int RS, bool INDEXED>
__global__ __launch_bounds__(256) void decode_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const float* __restrict__ g,
    const float* __restrict__ beta, float* __restrict__ state,
    uint16_t* __restrict__ o, int H_qk, int H_v, int blocks_per_head, float scale,
    const int32_t* __restrict__ idx, int P, int flags) {
    constexpr int F4_ROW = D / 4;
    constexpr int LPR = F4_ROW < 8 ? F4_ROW : 8;
    constexpr int J = F4_ROW / LPR;
    constexpr int RPI = 64 / LPR;
    constexpr int ROWS_PER_WAVE = RPI * RS;

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int nwave = blockDim.x >> 6;
    const int head = blockIdx.x / blocks_per_head;  // b * H_v + h
    const int blk = blockIdx.x - head * blocks_per_head;
    const int b = head / H_v;
    const int h = head - b * H_v;
    const int hq = h / (H_v / H_qk);
    long shead = head;  // (state slot) H_v + h
    if constexpr (INDEXED) {
        const int slot = idx[b];
        if (slot < 0 || slot >= P) return;
        shead = (long)slot * H_v + h;
    }
    const int row0 = (blk * nwave + wave) * ROWS_PER_WAVE;
    const int sub = lane / LPR;
    const int c = lane % LPR;

    // q and k slices for this lane's columns, widened to fp32 (L2-normalised
    // and rounded to bf16 again first, with the prologue flag).
    const uint16_t* kp = k + ((size_t)b * H_qk + hq) * D;
    const uint16_t* qp = q + ((size_t)b * H_qk + hq) * D;
    const bool norm = (flags & kFlagQkL2Norm) != 0;
    const float rk = norm ? row_inv_norm<D>(kp) : 1.f;
    const float rq = norm ? row_inv_norm<D>(qp) : 1.f;
    float kf[J][4], qf[J][4];
    float kq = 0.f;
#pragma unroll
    for (int j = 0; j < J; ++j) {
        const int col = (j * LPR + c) * 4;
        uint2 kk = *reinterpret_cast<const uint2*>(kp + col);
        uint2 qq = *reinterpret_cast<const uint2*>(qp + col);
        if (norm) {
            kk = uint2{scale_bf16x2(kk.x, rk), scale_bf16x2(kk.y, rk)};
            qq = uint2{scale_bf16x2(qq.x, rq), scale_bf16x2(qq.y, rq)};
        }
        kf[j][0] = bf16_to_f32(kk.x & 0xFFFF); kf[j][1] = bf16_to_f32(kk.x >> 16);
        kf[j][2] = bf16_to_f32(kk.y & 0xFFFF); kf[j][3] = bf16_to_f32(kk.y >> 16);
        qf[j][0] = bf16_to_f32(qq.x & 0xFFFF); qf[j][1] = bf16_to_f32(qq.x >> 16);
        qf[j][2] = bf16_to_f32(qq.y & 0xFFFF); qf[j][3] = bf16_to_f32(qq.y >> 16);
#pragma unroll
        for (int e = 0; e < 4; ++e) kq = fmaf(kf[j][e], qf[j][e], kq);
    }
    kq = group_sum<LPR>(kq);

    const bool logits = (flags & kFlagGateLogits) != 0;
    const float alpha = fast_exp(logits ? gate_from_logit(g[head]) : g[head]);
    const float bt = logits ? beta_from_logit(beta[head]) : beta[head];
    float* sp = state + (size_t)shead * D * D;
    const uint16_t* vp = v + (size_t)head * D;
    uint16_t* op = o + (size_t)head * D;

    // Issue every state load of this lane before any arithmetic.
    f32x4_t s[RS][J];
#pragma unroll
    for (int r = 0; r < RS; ++r) {
        const int row = row0 + r * RPI + sub;
#pragma unroll
        for (int j = 0; j < J; ++j)
            s[r][j] = __builtin_nontemporal_load(
                reinterpret_cast<const f32x4_t*>(sp + (size_t)row * D + (j * LPR + c) * 4));
    }
    float vi[RS];
#pragma unroll
    for (int r = 0; r < RS; ++r) vi[r] = bf16_to_f32(vp[row0 + r * RPI + sub]);

#pragma unroll
    for (int r = 0; r < RS; ++r) {
        const int row = row0 + r * RPI + sub;
        float kv = 0.f, sq = 0.f;
#pragma unroll
        for (int j = 0; j < J; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                kv = fmaf(s[r][j][e], kf[j][e], kv);
                sq = fmaf(s[r][j][e], qf[j][e], sq);
            }
        kv = group_sum<LPR>(kv);
        sq = group_sum<LPR>(sq);
        const float u = bt * (vi[r] - alpha * kv);
#pragma unroll
        for (int j = 0; j < J; ++j) {
            f32x4_t nv;
#pragma unroll
            for (int e = 0; e < 4; ++e) nv[e] = fmaf(alpha, s[r][j][e], u * kf[j][e]);
            __builtin_nontemporal_store(nv, reinterpret_cast<f32x4_t*>(sp + (size_t)row * D + (j * LPR + c) * 4));
        }
        if (c == 0) op[row] = f32_to_bf16(scale * fmaf(alpha, sq, u * kq));
    }
}

// Rows per workgroup = nwave * RS * (64 / LPR).  With D = 128 a workgroup of
// four waves covers 32 rows (16 KiB of state): of the tile shapes measured for
// in-place streaming with non-temporal loads and stores (8 to 64 KiB per
// workgroup), this one ran fastest.  Below 128 heads each workgroup is a single
// wave (8 rows) so that at least ~500 workgroups are in flight.
template <int D>
static hipError_t launch_decode_d(const DecodeArgs& a, hipStream_t stream) {
    constexpr int F4_ROW = D / 4;
    constexpr int LPR = F4_ROW < 8 ? F4_ROW : 8;
    constexpr int RPI = 64 / LPR;
    const long heads = (long)a.B * a.H_v;
    const int nwave = (D == 128 && heads >= 128) ? 4 : 1;
    const int rows_per_block = nwave * RPI;
    const int blocks_per_head = D / rows_per_block;
    const dim3 grid((unsigned)(heads * blocks_per_head));
    const dim3 block(64 * nwave);
    if (a.state_idx != nullptr)
        hipLaunchKernelGGL((decode_kernel<D, 1, true>), grid, block, 0, stream, (const uint16_t*)a.q,
                           (const uint16_t*)a.k, (const uint16_t*)a.v, a.g, a.beta, a.state,
                           (uint16_t*)a.o, a.H_qk, a.H_v, blocks_per_head, a.scale, a.state_idx, a.P, a.flags);
    else
        hipLaunchKernelGGL((decode_kernel<D, 1, false>), grid, block, 0, stream, (const uint16_t*)a.q,
                           (const uint16_t*)a.k, (const uint16_t*)a.v, a.g, a.beta, a.state,
                           (uint16_t*)a.o, a.H_qk, a.H_v, blocks_per_head, a.scale, nullptr, 0, a.flags);
    return hipGetLastError();
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
    if (a.D == 128) return launch_decode_d<128>(a, stream);
    return launch_decode_d<16>(a, stream);
}

}  // namespace gdn
