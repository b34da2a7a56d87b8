// Stable counting sort of the channels of one searched weight by chosen format, run by one
// workgroup of NT threads (the search's grouping launch, or a workgroup of the packing
// launch): thread t counts the formats of a run of consecutive channels (a multiple of
// 16, read 16 bytes at a time), an exclusive scan over the threads (per format) gives each
// run its start inside every group, and the thread then places its channels in order --
// into LDS when the caller provides room for the permutation (then copied out with
// coalesced 16-byte stores), else directly.
#ifndef CHAM_GROUP_H_
#define CHAM_GROUP_H_

#include "cham_device.h"

namespace cham {

constexpr int kGroupRun = 16;

struct GroupArgs {
    const uint8_t* fmt;
    int N;
    int32_t* perm;       // NULL = skip
    int32_t* group_off;  // NULL = skip
};

// 16 format bytes from channel c on; bytes at or past N read as 0xFF (no format)
CHAM_DEV uint4 fmt16(const uint8_t* fmt, int N, int c, bool aligned) {
    if (aligned && c + 16 <= N) return *reinterpret_cast<const uint4*>(fmt + c);
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint32_t v = 0u;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int r = c + 4 * i + b;
            v |= (r < N ? (uint32_t)fmt[r] : 0xFFu) << (8 * b);
        }
        w[i] = v;
    }
    return make_uint4(w[0], w[1], w[2], w[3]);
}

// lperm: LDS room for N entries, or nullptr (permutation written directly).  Every
// thread of the workgroup must call this.
template <int NT>
CHAM_DEV void group_channels(const GroupArgs& a, int32_t* lperm) {
    constexpr int NW = NT / kWave;
    __shared__ int32_t wtot[NW][CHAM_W_NFMT];
    __shared__ int32_t gbase[CHAM_W_NFMT];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int N = a.N;
    const bool aligned = ((uintptr_t)a.fmt & 15u) == 0;
    const int R = ((N + NT - 1) / NT + kGroupRun - 1) / kGroupRun * kGroupRun;
    const int64_t c0l = (int64_t)t * R;
    const int c0 = c0l < N ? (int)c0l : N, c1 = c0l + R < N ? (int)(c0l + R) : N;
    int32_t cnt[CHAM_W_NFMT];
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) cnt[f] = 0;
    // four 16-byte loads in flight, then their counts
    for (int c = c0; c < c1; c += 64) {
        uint4 q[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) q[i] = c + 16 * i < c1 ? fmt16(a.fmt, N, c + 16 * i, aligned) : make_uint4(~0u, ~0u, ~0u, ~0u);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t w[4] = {q[i].x, q[i].y, q[i].z, q[i].w};
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int f = (w[j >> 2] >> (8 * (j & 3))) & 255u;
#pragma unroll
                for (int g = 0; g < CHAM_W_NFMT; ++g) cnt[g] += f == g;
            }
        }
    }
    // exclusive scan over the threads, per format: within the wave, then across waves
    int32_t pre[CHAM_W_NFMT];
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) {
        int32_t v = cnt[f];
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int32_t u = __shfl_up(v, o, kWave);
            if (lane >= o) v += u;
        }
        pre[f] = v - cnt[f];
        if (lane == 63) wtot[wave][f] = v;
    }
    __syncthreads();
    if (t < CHAM_W_NFMT) {  // exclusive scan of the wave totals per format, in place
        int32_t acc = 0;
        for (int w = 0; w < NW; ++w) {
            const int32_t v = wtot[w][t];
            wtot[w][t] = acc;
            acc += v;
        }
        gbase[t] = acc;  // format total for now
    }
    __syncthreads();
    if (t == 0) {
        int32_t o = 0;
#pragma unroll
        for (int f = 0; f < CHAM_W_NFMT; ++f) {
            const int32_t tot = gbase[f];
            gbase[f] = o;
            if (a.group_off) a.group_off[f] = o;
            o += tot;
        }
        if (a.group_off) a.group_off[CHAM_W_NFMT] = o;
    }
    __syncthreads();
    if (!a.perm) return;
    int32_t* dst = lperm ? lperm : a.perm;
#pragma unroll
    for (int f = 0; f < CHAM_W_NFMT; ++f) pre[f] += gbase[f] + wtot[wave][f];
    for (int c = c0; c < c1; c += 16) {
        const uint4 q = fmt16(a.fmt, N, c, aligned);
        const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int f = (w[j >> 2] >> (8 * (j & 3))) & 255u;
            int32_t pos = -1;
#pragma unroll
            for (int g = 0; g < CHAM_W_NFMT; ++g) {
                if (f == g) pos = pre[g]++;
            }
            if (pos >= 0) dst[pos] = c + j;
        }
    }
    if (!lperm) return;
    __syncthreads();  // every channel has a format of the palette, so all N slots are set
    if (((uintptr_t)a.perm & 15u) == 0) {
        const int n4 = N >> 2;
        for (int i = t; i < n4; i += NT)
            reinterpret_cast<int4*>(a.perm)[i] = reinterpret_cast<const int4*>(lperm)[i];
        for (int i = (n4 << 2) + t; i < N; i += NT) a.perm[i] = lperm[i];
    } else {
        for (int i = t; i < N; i += NT) a.perm[i] = lperm[i];
    }
}

}  // namespace cham

#endif  // CHAM_GROUP_H_
