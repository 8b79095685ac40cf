// Attention-accumulated modality score (Sec. 3.2.1, Eq. 2-4).
//
// attn_fwd_kernel: causal softmax attention inside each sample, one
// workgroup per (128 query rows, query head), with the modality scores of the
// keys carried along as two extra value channels (the supplementary
// implementation note) — here in fp32 on the vector ALUs next to the bf16
// MFMA product of the values, so the aggregated scores keep fp32 accuracy.
// Outputs: O[T][H][d_head] = Attn_h V (bf16) and m_heads[T][H][2] = Attn_h M
// (Eq. 3 per head). attn_update_kernel averages m_heads over heads (Eq. 3)
// and applies the norm-weighted residual mix (Eq. 4). attn_init_kernel
// writes the one-hot layer-0 scores (Eq. 2).
//
// Layout of the attention (per wave, 32 queries; per key block, 64 keys):
//   S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (A = K rows from LDS, B = the
//   wave's Q rows held in registers): accumulator element v of lane l is key
//   8*(v/4) + 4*(l/32) + v%4 of the 32-key tile and query l%32, so softmax
//   statistics are per lane plus one exchange with lane l ^ 32.
//   O^T += V^T P^T: P^T's B operand is the S^T accumulator itself, read in
//   the order above; V stays row-major in LDS and the A operand (4 keys of one
//   dim per 8 bytes) comes from the transposing LDS read ds_read_b64_tr_b16:
//   within each 16-lane group, lane j supplies the address of key j/4 and
//   dims 4*(j%4) .. + 3 and receives dim j of those four keys.
// The running maximum is rescaled lazily (only when a block's maximum exceeds
// it by more than 8 in log2 units); blocks that every query of a wave sees
// whole skip the mask.
// Logits use exp2 with the scale folded into log2(e).
#include "common.h"
#include "kernels.h"

namespace smoes {

namespace {

constexpr int AT_BQ = 128;  // query rows per workgroup (4 waves x 32)
constexpr int AT_BK = 64;   // keys per block
constexpr int AT_THREADS = 256;
constexpr int kAtBufFlags = 0x00020000;
constexpr uint32_t kAtOob = 0x80000000u;  // a byte offset past any buffer: reads return 0

typedef int at_i32x4 __attribute__((ext_vector_type(4)));
typedef short at_v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) at_v4i16 at_lds_v4i16;

// Start of the sample that holds token q: offsets[s] for the largest s < n_batch
// with offsets[s] <= q.
__device__ __forceinline__ int sample_start(const int32_t* __restrict__ offsets, int n_batch, int q) {
    int lo = 0, hi = n_batch - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (offsets[mid] <= q) lo = mid; else hi = mid - 1;
    }
    return offsets[lo];
}

typedef float at_f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 at_bf16x2 __attribute__((ext_vector_type(2)));

// Two floats to two bf16 (round to nearest even; one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(at_f32x2{a, b}, at_bf16x2));
}

template <int DH>
__device__ __forceinline__ void attn_fwd_body(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                                              const uint16_t* __restrict__ v, int64_t T, int H, int Hkv,
                                              const int32_t* __restrict__ offsets, int n_batch,
                                              const float* __restrict__ m_in, float scale_log2,
                                              uint16_t* __restrict__ o, float* __restrict__ m_heads) {
    constexpr int CPK = DH / 8;           // 16-byte chunks per key row
    constexpr int KC = DH / 16;           // K = 16 slices of the QK^T contraction
    constexpr int DT = DH / 32;           // 32-row tiles of O^T
    constexpr int KCH = AT_BK * CPK / AT_THREADS;  // K (and V) 16-byte chunks per thread per block
    static_assert(KCH >= 1, "head size");
    // Padded rows instead of swizzles, so that every fragment address is a
    // per-lane base plus an immediate. Pitches chosen so that the fragment
    // reads hit distinct LDS banks: K rows of DH + 8 elements (16-byte reads of
    // 16 consecutive keys), V rows of DH + 32 elements (the transposing reads
    // of 8 keys x 64 bytes).
    constexpr int KP = DH + 8;   // K row pitch (elements)
    constexpr int VP = DH + 32;  // V row pitch (elements)
    __shared__ __attribute__((aligned(16))) uint16_t k_lds[AT_BK * KP];
    __shared__ __attribute__((aligned(16))) uint16_t v_lds[AT_BK * VP];
    __shared__ __attribute__((aligned(16))) float mv_lds[2][AT_BK];

    const int nqb = static_cast<int>(ceil_div(T, AT_BQ));
    const int hq = blockIdx.y;
    // Two workgroups share a CU: those L and L + N / 2 in dispatch order (N =
    // all of them), i.e. heads h and h + H / 2 at the same blockIdx.x. The
    // lower half of the heads takes the query blocks from the last (longest
    // causal range) down, the upper half from the first up, so a CU holds a
    // long and a short block rather than two of the same length.
    const int qb = 2 * hq < static_cast<int>(gridDim.y) ? nqb - 1 - static_cast<int>(blockIdx.x)
                                                      : static_cast<int>(blockIdx.x);
    const int hk = hq / (H / Hkv);
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int half = lane >> 5, l32 = lane & 31;
    const int Ti = static_cast<int>(T);
    const int row0 = qb * AT_BQ;
    // first key any row of the block may see (clamped so that malformed offsets cannot run the loop away)
    const int kstart = min(max(sample_start(offsets, n_batch, row0), 0), row0);
    const int kend = min(row0 + AT_BQ, Ti);
    const int qi = row0 + wave * 32 + l32;
    const bool q_ok = qi < Ti;
    const int qe = q_ok ? qi : Ti - 1;
    const int qstart = min(max(sample_start(offsets, n_batch, qe), 0), qe);
    const int wq0 = row0 + wave * 32;  // first query row of this wave
    // per-lane base of the transposing V reads: 16-lane group g = lane / 16
    // covers dims 16 (g & 1) .. + 15 of a 32-dim tile and keys 4 (g >> 1) .. + 3
    // of an 8-key half-slice; lane j of the group points at key j / 4, dims 4 (j % 4) ..
    const int vtr_base = ((lane >> 5) * 4 + ((lane & 15) >> 2)) * VP + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    // sample start of the wave's last query: the largest start of its queries
    const int wq_start_max = __builtin_amdgcn_readlane(qstart, 31);

    const __amdgpu_buffer_rsrc_t rsK = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(k), 0, static_cast<int>(T * Hkv * DH * 2), kAtBufFlags);
    const __amdgpu_buffer_rsrc_t rsV = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(v), 0, static_cast<int>(T * Hkv * DH * 2), kAtBufFlags);
    const __amdgpu_buffer_rsrc_t rsM = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(m_in), 0, static_cast<int>(T * 2 * 4), kAtBufFlags);

    // the wave's Q rows as B fragments held in registers for the whole key
    // loop: slice c = dims 16c + 8*half .. + 7 of query qe
    at_i32x4 qf[KC];
    {
        const uint4* qrow = reinterpret_cast<const uint4*>(q + (static_cast<int64_t>(qe) * H + hq) * DH);
#pragma unroll
        for (int c = 0; c < KC; ++c) {
            const uint4 t = qrow[2 * c + half];
            qf[c] = at_i32x4{static_cast<int>(t.x), static_cast<int>(t.y), static_cast<int>(t.z), static_cast<int>(t.w)};
        }
    }

    // global -> register staging of one key block
    // byte offset of the row of `key` in K or V; keys below 0 wrap to offsets
    // >= 2^31 and keys >= T land past the buffer: the bounds check reads zeros
    auto key_off = [&](int key) -> uint32_t {
        return static_cast<uint32_t>((key * Hkv + hk) * DH * 2);
    };
    at_i32x4 kr[KCH], vr[KCH];
    float2 mr;
    auto load_block = [&](int kb0_) {
        int kb0 = kb0_;
        asm volatile("" : "+v"(kb0));  // per-lane copy: the per-item offsets are rebuilt in the loop
#pragma unroll
        for (int i = 0; i < KCH; ++i) {
            const int id = threadIdx.x + i * AT_THREADS;
            const int key = id / CPK, c = id % CPK;
            kr[i] = __builtin_amdgcn_raw_buffer_load_b128(rsK, static_cast<int>(key_off(kb0 + key) + c * 16), 0, 0);
        }
#pragma unroll
        for (int i = 0; i < KCH; ++i) {
            const int id = threadIdx.x + i * AT_THREADS;
            const int key = id / CPK, c = id % CPK;
            vr[i] = __builtin_amdgcn_raw_buffer_load_b128(rsV, static_cast<int>(key_off(kb0 + key) + c * 16), 0, 0);
        }
        if (threadIdx.x < AT_BK) {
            const int key = kb0 + static_cast<int>(threadIdx.x);
            const uint32_t off = (key >= 0 && key < Ti) ? static_cast<uint32_t>(key * 8) : kAtOob;
            mr.x = __int_as_float(__builtin_amdgcn_raw_buffer_load_b32(rsM, static_cast<int>(off), 0, 0));
            mr.y = __int_as_float(__builtin_amdgcn_raw_buffer_load_b32(rsM, static_cast<int>(off == kAtOob ? off : off + 4), 0, 0));
        }
    };
    // register -> LDS: K and V rows (16-byte chunks, padded rows)
    auto store_block = [&]() {
        int sz = 0;  // opaque zero: keeps the store addresses from being hoisted out of the key loop
        asm volatile("" : "+v"(sz));
        uint16_t* kst = k_lds + sz;
        uint16_t* vst = v_lds + sz;
#pragma unroll
        for (int i = 0; i < KCH; ++i) {
            const int id = threadIdx.x + i * AT_THREADS;
            const int key = id / CPK, c = id % CPK;
            *reinterpret_cast<at_i32x4*>(kst + key * KP + c * 8) = kr[i];
            *reinterpret_cast<at_i32x4*>(vst + key * VP + c * 8) = vr[i];
        }
        if (threadIdx.x < AT_BK) {
            mv_lds[0][threadIdx.x] = mr.x;
            mv_lds[1][threadIdx.x] = mr.y;
        }
    };

    f32x16_t oacc[DT];
#pragma unroll
    for (int i = 0; i < DT; ++i) oacc[i] = f32x16_t{};
    float m_run = -INFINITY, l_run = 0.f, a0 = 0.f, a1 = 0.f;

    const int nkb = static_cast<int>(ceil_div(kend - kstart, AT_BK));
    load_block(kstart);
    for (int b = 0; b < nkb; ++b) {
        const int kb0 = kstart + b * AT_BK;
        __syncthreads();  // the previous block's LDS reads are done
        store_block();
        __syncthreads();
        if (b + 1 < nkb) load_block(kb0 + AT_BK);  // next block's loads fly during this block's math
        // LDS addresses are rebuilt inside the loop from an opaque zero: hoisting
        // all of them out of the loop would not fit the register budget
        int lz = 0;
        asm volatile("" : "+v"(lz));
        const uint16_t* kl = k_lds + lz;
        const uint16_t* vl = v_lds + lz;
        const float* ml = &mv_lds[0][0] + lz;

        // S^T = K Q^T for the two 32-key tiles; K fragments read one slice ahead
        // (the scheduling barriers keep the compiler from hoisting every LDS
        // read of the block, which would not fit the register budget)
        f32x16_t s[2] = {f32x16_t{}, f32x16_t{}};
        auto kfrag = [&](int c, int t) {
            const int key = t * 32 + l32;
            return *reinterpret_cast<const bf16x8_t*>(kl + key * KP + (2 * c + half) * 8);
        };
        bf16x8_t ka[2][2];
        ka[0][0] = kfrag(0, 0);
        ka[0][1] = kfrag(0, 1);
#pragma unroll
        for (int c = 0; c < KC; ++c) {
            if (c + 1 < KC) {
                ka[(c + 1) & 1][0] = kfrag(c + 1, 0);
                ka[(c + 1) & 1][1] = kfrag(c + 1, 1);
            }
#pragma unroll
            for (int t = 0; t < 2; ++t)
                s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[c & 1][t], __builtin_bit_cast(bf16x8_t, qf[c]), s[t], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
        // The block maximum of this query's logits; keys outside the query's
        // sample or past its diagonal are masked, except in blocks that every
        // query of the wave sees whole (the common case, checked per wave).
        const bool full = kb0 >= wq_start_max && kb0 + AT_BK - 1 <= wq0;
        float mx = -INFINITY;
        if (full) {
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[t][e]);
        } else {
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int key = kb0 + t * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
                    const float x = (key >= qstart && key <= qe) ? s[t][e] : -INFINITY;
                    s[t][e] = x;
                    mx = fmaxf(mx, x);
                }
        }
        const float mblk = fmaxf(mx, __shfl_xor(mx, 32, kWave)) * scale_log2;
        // Lazy rescaling: the reference m_run moves only when a block's maximum
        // exceeds it by more than 8 (log2 units), so exp2 stays below 2^8 and
        // the accumulators are rescaled in few blocks. Both halves of a query
        // take the same decision.
        const bool grow = mblk > m_run + 8.f;
        if (__builtin_amdgcn_ballot_w64(grow) != 0) {
            const float m_new = grow ? mblk : m_run;
            const float alpha = grow ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.f;  // m_run = -inf: 0
            m_run = m_new;
            l_run *= alpha;
            a0 *= alpha;
            a1 *= alpha;
#pragma unroll
            for (int i = 0; i < DT; ++i) oacc[i] *= alpha;
        }
        const float m_use = m_run == -INFINITY ? 0.f : m_run;
        float ls = 0.f, s0 = 0.f, s1 = 0.f;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                __builtin_amdgcn_sched_barrier(0);
                const int kk = t * 32 + 8 * g + 4 * half;  // four consecutive keys of this lane
                const float4 mv = *reinterpret_cast<const float4*>(ml + kk);
                const float4 mt = *reinterpret_cast<const float4*>(ml + AT_BK + kk);
                const float mva[4] = {mv.x, mv.y, mv.z, mv.w}, mta[4] = {mt.x, mt.y, mt.z, mt.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float p = __builtin_amdgcn_exp2f(fmaf(s[t][4 * g + e], scale_log2, -m_use));
                    s[t][4 * g + e] = p;
                    ls += p;
                    s0 = fmaf(p, mva[e], s0);
                    s1 = fmaf(p, mta[e], s1);
                }
            }
        l_run += ls;
        a0 += s0;
        a1 += s1;
        // O^T += V^T P^T over four 16-key slices
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const f32x16_t& st = s[c >> 1];
            const int e0 = 8 * (c & 1);
            const at_i32x4 pb{static_cast<int>(pack_bf16x2(st[e0 + 0], st[e0 + 1])),
                              static_cast<int>(pack_bf16x2(st[e0 + 2], st[e0 + 3])),
                              static_cast<int>(pack_bf16x2(st[e0 + 4], st[e0 + 5])),
                              static_cast<int>(pack_bf16x2(st[e0 + 6], st[e0 + 7]))};
#pragma unroll
            for (int i = 0; i < DT; ++i) {
                // keys 16c + 4 half + 0..3 and 16c + 8 + 4 half + 0..3 of dim 32i + lane % 32
                const at_v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (at_lds_v4i16*)(vl + vtr_base + (16 * c) * VP + 32 * i));
                const at_v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (at_lds_v4i16*)(vl + vtr_base + (16 * c + 8) * VP + 32 * i));
                const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
                const at_i32x4 va{static_cast<int>(l2.x), static_cast<int>(l2.y), static_cast<int>(h2.x), static_cast<int>(h2.y)};
                oacc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, va),
                                                                  __builtin_bit_cast(bf16x8_t, pb), oacc[i], 0, 0, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    // both halves of the wave hold partial sums of the same query
    const float l_tot = l_run + __shfl_xor(l_run, 32, kWave);
    const float a0t = a0 + __shfl_xor(a0, 32, kWave);
    const float a1t = a1 + __shfl_xor(a1, 32, kWave);
    if (!q_ok) return;
    const float inv = 1.f / l_tot;
    uint16_t* orow = o + (static_cast<int64_t>(qi) * H + hq) * DH;
#pragma unroll
    for (int i = 0; i < DT; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int d0 = i * 32 + 8 * g + 4 * half;
            *reinterpret_cast<uint2*>(orow + d0) =
                make_uint2(pack_bf16x2(oacc[i][4 * g] * inv, oacc[i][4 * g + 1] * inv),
                           pack_bf16x2(oacc[i][4 * g + 2] * inv, oacc[i][4 * g + 3] * inv));
        }
    if (half == 0) {
        float* mh = m_heads + (static_cast<int64_t>(qi) * H + hq) * 2;
        mh[0] = a0t / l_tot;
        mh[1] = a1t / l_tot;
    }
}

__global__ void __launch_bounds__(AT_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
attn_fwd_kernel_d128(const uint16_t* q, const uint16_t* k, const uint16_t* v, int64_t T, int H, int Hkv,
                     const int32_t* offsets, int n_batch, const float* m_in, float scale_log2, uint16_t* o,
                     float* m_heads) {
    attn_fwd_body<128>(q, k, v, T, H, Hkv, offsets, n_batch, m_in, scale_log2, o, m_heads);
}

__global__ void __launch_bounds__(AT_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
attn_fwd_kernel_d64(const uint16_t* q, const uint16_t* k, const uint16_t* v, int64_t T, int H, int Hkv,
                    const int32_t* offsets, int n_batch, const float* m_in, float scale_log2, uint16_t* o,
                    float* m_heads) {
    attn_fwd_body<64>(q, k, v, T, H, Hkv, offsets, n_batch, m_in, scale_log2, o, m_heads);
}

// Eq. 3 head average and Eq. 4 mix: one wave per token.
template <bool BF16>
__global__ void __launch_bounds__(256) attn_update_kernel(const void* __restrict__ x, const void* __restrict__ x_attn,
                                                          int64_t T, int d, const float* __restrict__ m_heads, int H,
                                                          const float* m_in, float* m_out) {
    const int64_t j = static_cast<int64_t>(blockIdx.x) * 4 + threadIdx.x / kWave;
    if (j >= T) return;
    const int lane = lane_id();
    float sx = 0.f, sa = 0.f;
    for (int c = lane * 8; c < d; c += kWave * 8) {
        float a[8], b[8];
        load8<BF16>(x, j * d + c, a);
        load8<BF16>(x_attn, j * d + c, b);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            sx += a[e] * a[e];
            sa += b[e] * b[e];
        }
    }
    sx = wave_sum_u(sx);
    sa = wave_sum_u(sa);
    if (lane != 0) return;
    const float nx = sqrtf(sx), na = sqrtf(sa);
    float t0 = 0.f, t1 = 0.f;
    for (int h = 0; h < H; ++h) {
        t0 += m_heads[(j * H + h) * 2];
        t1 += m_heads[(j * H + h) * 2 + 1];
    }
    const float invh = 1.f / static_cast<float>(H);
    const float m0 = m_in[j * 2], m1 = m_in[j * 2 + 1];
    const float den = nx + na;
    float r0 = m0, r1 = m1;
    if (den > 0.f) {
        r0 = (na * (t0 * invh) + nx * m0) / den;
        r1 = (na * (t1 * invh) + nx * m1) / den;
    }
    m_out[j * 2] = r0;
    m_out[j * 2 + 1] = r1;
}

__global__ void attn_init_kernel(const uint8_t* __restrict__ modality_id, int64_t T, float* __restrict__ M) {
    for (int64_t j = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; j < T;
         j += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const uint8_t m = modality_id[j];
        M[2 * j] = m == 0 ? 1.f : 0.f;
        M[2 * j + 1] = m == 1 ? 1.f : 0.f;
    }
}

}  // namespace

hipError_t launch_attention(const void* q, const void* k, const void* v, int64_t T, int H, int Hkv, int head_dim,
                            const int32_t* sample_offsets, int n_batch, const float* m_in, float scale, void* o,
                            float* m_heads, hipStream_t stream) {
    if (T == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>(ceil_div(T, AT_BQ)), static_cast<unsigned>(H));
    const float scale_log2 = scale * 1.4426950408889634f;
    if (head_dim == 128)
        hipLaunchKernelGGL(attn_fwd_kernel_d128, grid, dim3(AT_THREADS), 0, stream, static_cast<const uint16_t*>(q),
                           static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), T, H, Hkv,
                           sample_offsets, n_batch, m_in, scale_log2, static_cast<uint16_t*>(o), m_heads);
    else
        hipLaunchKernelGGL(attn_fwd_kernel_d64, grid, dim3(AT_THREADS), 0, stream, static_cast<const uint16_t*>(q),
                           static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), T, H, Hkv,
                           sample_offsets, n_batch, m_in, scale_log2, static_cast<uint16_t*>(o), m_heads);
    return hipGetLastError();
}

hipError_t launch_attn_update(const void* x, const void* x_attn, int act_dtype, int64_t T, int d,
                              const float* m_heads, int H, const float* m_in, float* m_out, hipStream_t stream) {
    if (T == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>(ceil_div(T, 4)));
    if (act_dtype == 1)
        hipLaunchKernelGGL(attn_update_kernel<true>, grid, dim3(256), 0, stream, x, x_attn, T, d, m_heads, H, m_in, m_out);
    else
        hipLaunchKernelGGL(attn_update_kernel<false>, grid, dim3(256), 0, stream, x, x_attn, T, d, m_heads, H, m_in, m_out);
    return hipGetLastError();
}

hipError_t launch_attn_init(const uint8_t* modality_id, int64_t T, float* M, hipStream_t stream) {
    if (T == 0) return hipSuccess;
    const int64_t b = ceil_div(T, 256);
    hipLaunchKernelGGL(attn_init_kernel, dim3(static_cast<unsigned>(b < 4096 ? b : 4096)), dim3(256), 0, stream,
                       modality_id, T, M);
    return hipGetLastError();
}

}  // namespace smoes
