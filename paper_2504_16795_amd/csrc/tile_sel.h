// Selections of a tile of consecutive query tokens (one (b, g), all inside one query
// chunk), prepared in LDS for the tile-major kernels (forward, query pass of the backward).
//
// The selection of token t is idx[t][0..k), w[t][0..k) (Sec. 3.1.1: the top-k chunks and
// their softmax weights).  Entries outside the token's candidates [0, ncand) are empty.
// The tables built here let every lane of a row block walk its token's chunks in the same
// descending order in which the tile's union of chunks is staged.
#pragma once

#include "mfma_common.h"

namespace hsa {

struct TileSel {
    int32_t* oidx;    // [TQ k] per slot: the chunk, -1 when empty
    float* ow;        // [TQ k] per slot: the weight, 0 when empty
    int32_t* sidx;    // [TQ k] per token: its distinct chunks in descending order, -1 pad
    uint8_t* sslot;   // [TQ k]   ... the first slot holding each
    float* sw;        // [TQ k]   ... the summed weight of the slots holding it
    uint32_t* ubits;  // [ceil(ncand / 32)] scratch bitmap
    int32_t* ulist;   // [TQ k] union of the tile's chunks, descending
    int* wsum;        // [NT / 64] scratch
};

// Builds the tables; every thread of the workgroup (NT threads) calls it.  sel0 is the
// element offset of token t0's slot 0 in idx / w, tstride the offset between tokens,
// ntok <= TQ the tokens of the tile inside the sequence.  Returns the union size; the
// tables are visible to all threads on return.
template <int NT, int TQ>
__device__ __forceinline__ int tile_selection(const TileSel& ts, const int32_t* __restrict__ idx,
                                              const float* __restrict__ w, size_t sel0,
                                              size_t tstride, int k, int ntok, int ncand) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int ne = TQ * k;
    const int nwd = (ncand + 31) >> 5;
    // 1. all slots of the tile in parallel
    for (int e = tid; e < ne; e += NT) {
        const int tau = e / k, s = e - tau * k;
        int c = -1;
        float wv = 0.f;
        if (tau < ntok) {
            const size_t o = sel0 + (size_t)tau * tstride + s;
            c = idx[o];
            wv = w[o];
            if (c < 0 || c >= ncand) {
                c = -1;
                wv = 0.f;
            }
        }
        ts.oidx[e] = c;
        ts.ow[e] = wv;
    }
    for (int i = tid; i < nwd; i += NT) ts.ubits[i] = 0u;
    __syncthreads();
    // 2. keys: the first slot holding a chunk keeps it, repeats and empty slots get -1
    //    (ulist serves as the key array until the union is listed)
    int32_t* key = ts.ulist;
    for (int e = tid; e < ne; e += NT) {
        const int tau = e / k, s = e - tau * k;
        const int32_t* oc = &ts.oidx[tau * k];
        const int c = oc[s];
        bool first = c >= 0;
        for (int s2 = 0; s2 < s && first; ++s2) first = oc[s2] != c;
        key[e] = first ? c : -1;
    }
    __syncthreads();
    // 3. rank of each key among the token's keys (descending); empty keys fill the tail
    for (int e = tid; e < ne; e += NT) {
        const int tau = e / k, s = e - tau * k;
        const int32_t* kt = &key[tau * k];
        const int c = kt[s];
        int pos = 0;
        float wm = 0.f;
        if (c >= 0) {
            for (int s2 = 0; s2 < k; ++s2) {
                pos += kt[s2] > c;
                if (ts.oidx[tau * k + s2] == c) wm += ts.ow[tau * k + s2];
            }
            atomicOr(&ts.ubits[c >> 5], 1u << (c & 31));
        } else {
            int nvalid = 0, before = 0;
            for (int s2 = 0; s2 < k; ++s2) {
                nvalid += kt[s2] >= 0;
                before += (s2 < s) && (kt[s2] < 0);
            }
            pos = nvalid + before;
        }
        ts.sidx[tau * k + pos] = c;
        ts.sslot[tau * k + pos] = (uint8_t)(c >= 0 ? s : 0);
        ts.sw[tau * k + pos] = wm;
    }
    __syncthreads();
    // 4. union in descending chunk order: thread i takes bitmap word nwd - 1 - i
    int total = 0;
    for (int w0 = 0; w0 < nwd; w0 += NT) {
        const int wi = nwd - 1 - (w0 + tid);
        const uint32_t word = (wi >= 0) ? ts.ubits[wi] : 0u;
        const int cnt = __popc(word);
        int incl = cnt;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int v = __shfl_up(incl, o, 64);
            if (lane >= o) incl += v;
        }
        if (lane == 63) ts.wsum[wave] = incl;
        __syncthreads();
        int pos = total;
        for (int i = 0; i < wave; ++i) pos += ts.wsum[i];
        pos += incl - cnt;
        uint32_t x = word;
        while (x) {
            const int bit = 31 - __clz(x);
            ts.ulist[pos++] = wi * 32 + bit;
            x &= ~(1u << bit);
        }
        for (int i = 0; i < NT / 64; ++i) total += ts.wsum[i];
        __syncthreads();
    }
    return total;
}

}  // namespace hsa
