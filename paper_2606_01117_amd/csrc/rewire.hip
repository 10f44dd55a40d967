// Group-shared rewiring of the supports (Alg. 3), the discrete phase of training:
//   1. score each (group k, slot j) by the |w| of the group's labels at that slot (fp32 sum over
//      the G labels in order: the algorithm's mean divides every score by the same G);
//   2. prune the m = floor(K F rho) smallest scores over all groups, ties to the lower flat index;
//   3. give each pruned slot a feature drawn uniformly from those its group does not keep (slots
//      in ascending order, each draw excluding the earlier ones), then re-sort the row, carrying
//      every slot's weight column (and velocity) with it;
//   4. reinitialise the pruned slots' weights: zero, or uniform in [-1/sqrt(F), 1/sqrt(F)].
// Draws come from SplitMix64 (Steele, Lea and Flood, 2014) in counter form: draw k F + j for the
// new feature of slot j of group k, draw K F + l F + j for label l's new weight at slot j.
#include "common.hpp"

namespace {

__device__ __forceinline__ uint64_t splitmix64_at(uint64_t s, uint64_t i) {
    uint64_t z = s + (i + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// Selection state of the radix select: the prefix of the threshold's key found so far, the bits it
// covers, and the rank of the wanted key among the keys that share the prefix.
struct RwState {
    uint32_t prefix, pmask;
    uint64_t rank;
};

// keys[k F + j] = bits of the fp32 sum over the group's labels of |W[l, j]| (non-negative, so the
// bit patterns order as the values)
template <typename T>
__global__ __launch_bounds__(256) void k_rw_scores(const T *__restrict__ W, int64_t K, int G, int F,
                                                   uint32_t *__restrict__ keys) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= K * F) return;
    const int64_t k = i / F;
    const int j = (int)(i - k * F);
    // the labels' weights 8 at a time, all 8 loads in flight before they are summed in order
    float s = 0.0f;
    const T *w = W + k * G * F + j;
    int g = 0;
    for (; g + 8 <= G; g += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = load_f32(w, (int64_t)(g + u) * F);
#pragma unroll
        for (int u = 0; u < 8; ++u) s += fabsf(v[u]);
    }
    for (; g < G; ++g) s += fabsf(load_f32(w, (int64_t)g * F));
    keys[i] = __float_as_uint(s);
}

__global__ void k_rw_init(uint32_t *__restrict__ hist, RwState *__restrict__ st, uint64_t rank) {
    const int t = threadIdx.x;
    if (t < 256) hist[t] = 0u;
    if (t == 0) *st = RwState{0u, 0u, rank};
}

// histogram of the next 8-bit digit (at `shift`) of the keys that share the current prefix
__global__ __launch_bounds__(256) void k_rw_hist(const uint32_t *__restrict__ keys, int64_t n,
                                                 const RwState *__restrict__ st, int shift,
                                                 uint32_t *__restrict__ hist) {
    __shared__ uint32_t h[256];
    h[threadIdx.x] = 0u;
    __syncthreads();
    const uint32_t prefix = st->prefix, pmask = st->pmask;
    // four keys per 16-byte load, four loads in flight per thread (the keys array is 256-byte
    // aligned); the last n mod 4 keys one by one
    const uint4 *k4 = reinterpret_cast<const uint4 *>(keys);
    const int64_t n4 = n / 4, stride = (int64_t)gridDim.x * blockDim.x;
    auto count = [&](uint32_t key) {
        if ((key & pmask) == prefix) atomicAdd(&h[(key >> shift) & 255u], 1u);
    };
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += 4 * stride) {
        uint4 v[4];
        bool ok[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            ok[u] = i + u * stride < n4;
            v[u] = ok[u] ? k4[i + u * stride] : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (ok[u]) {
                count(v[u].x);
                count(v[u].y);
                count(v[u].z);
                count(v[u].w);
            }
    }
    if (blockIdx.x == 0 && threadIdx.x < n - 4 * n4) count(keys[4 * n4 + threadIdx.x]);
    __syncthreads();
    if (h[threadIdx.x]) atomicAdd(&hist[threadIdx.x], h[threadIdx.x]);
}

// pick the digit whose cumulative count passes the wanted rank; clear the histogram for the next pass
__global__ void k_rw_pick(uint32_t *__restrict__ hist, RwState *__restrict__ st, int shift) {
    __shared__ uint32_t h[256];
    const int t = threadIdx.x;
    h[t] = hist[t];
    hist[t] = 0u;
    __syncthreads();
    if (t == 0) {
        RwState s = *st;
        uint64_t cum = 0;
        int d = 255;
        for (int b = 0; b < 256; ++b) {
            if (cum + h[b] > s.rank) {
                d = b;
                break;
            }
            cum += h[b];
        }
        s.rank -= cum;
        s.prefix |= (uint32_t)d << shift;
        s.pmask |= 255u << shift;
        *st = s;
    }
}

constexpr int kRwBlock = 1024;   // keys per block of the tie scan (256 threads x 4)

// number of keys equal to the threshold per block of kRwBlock keys
__global__ __launch_bounds__(256) void k_rw_eqcount(const uint32_t *__restrict__ keys, int64_t n,
                                                    const RwState *__restrict__ st, uint32_t *__restrict__ cnt) {
    __shared__ uint32_t tot;
    if (threadIdx.x == 0) tot = 0u;
    __syncthreads();
    const uint32_t T = st->prefix;
    const int64_t i0 = (int64_t)blockIdx.x * kRwBlock + 4 * threadIdx.x;
    uint32_t c = 0;
    for (int e = 0; e < 4; ++e) c += (i0 + e < n && keys[i0 + e] == T) ? 1u : 0u;
    if (c) atomicAdd(&tot, c);
    __syncthreads();
    if (threadIdx.x == 0) cnt[blockIdx.x] = tot;
}

// exclusive prefix of the per-block counts, in block order (one workgroup of 1024 threads): each
// thread sums a contiguous run of counts, one scan of the 1024 run sums, then each thread writes
// its run's prefixes (integer sums: the same values in any order)
constexpr int kRwScanThreads = 1024;
__global__ __launch_bounds__(kRwScanThreads) void k_rw_scan(uint32_t *__restrict__ cnt, int64_t nb) {
    __shared__ uint32_t part[kRwScanThreads];
    const int t = threadIdx.x;
    const int64_t per = (nb + kRwScanThreads - 1) / kRwScanThreads;
    const int64_t b = t * per, e = b + per < nb ? b + per : nb;
    uint32_t sum = 0u;
#pragma unroll 8
    for (int64_t i = b; i < e; ++i) sum += cnt[i];
    part[t] = sum;
    __syncthreads();
    for (int off = 1; off < kRwScanThreads; off <<= 1) {   // inclusive Hillis-Steele scan
        const uint32_t a = t >= off ? part[t - off] : 0u;
        __syncthreads();
        part[t] += a;
        __syncthreads();
    }
    uint32_t run = part[t] - sum;
    for (int64_t i = b; i < e; ++i) {
        const uint32_t v = cnt[i];
        cnt[i] = run;
        run += v;
    }
}

// mask[i] = key < T, or key == T and fewer than `need` equal keys precede it
__global__ __launch_bounds__(256) void k_rw_mark(const uint32_t *__restrict__ keys, int64_t n,
                                                 const RwState *__restrict__ st, const uint32_t *__restrict__ pre,
                                                 uint8_t *__restrict__ mask) {
    __shared__ uint32_t part[256];
    const uint32_t T = st->prefix;
    const uint64_t need = st->rank + 1;   // the wanted key is the rank-th (0-based) among those equal to T
    const int64_t i0 = (int64_t)blockIdx.x * kRwBlock + 4 * threadIdx.x;
    uint32_t key[4], c = 0;
    for (int e = 0; e < 4; ++e) {
        key[e] = i0 + e < n ? keys[i0 + e] : 0xFFFFFFFFu;
        c += (i0 + e < n && key[e] == T) ? 1u : 0u;
    }
    part[threadIdx.x] = c;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const uint32_t a = threadIdx.x >= off ? part[threadIdx.x - off] : 0u;
        __syncthreads();
        part[threadIdx.x] += a;
        __syncthreads();
    }
    uint64_t r = (uint64_t)pre[blockIdx.x] + part[threadIdx.x] - c;   // equal keys before this thread's
    for (int e = 0; e < 4; ++e) {
        if (i0 + e >= n) break;
        uint8_t mk = key[e] < T ? 1 : 0;
        if (key[e] == T) mk = r++ < need ? 1 : 0;
        mask[i0 + e] = mk;
    }
}

// Regrowth, one wave per group with a pruned slot.  F <= 256 slots (up to four per lane), H <= 1024
// features (one 32-bit word of the wave's used-feature bitmap per lane).
constexpr int kRwWaves = 4;
constexpr int kRwMaxF = 256;

// NPL: 64-slot words of a support (F <= 64 NPL)
template <typename T, int NPL>
__global__ __launch_bounds__(64 * kRwWaves) void k_rw_regrow(int32_t *__restrict__ idx, T *__restrict__ W,
                                                             float *__restrict__ mom, const uint8_t *__restrict__ mask,
                                                             int64_t K, int G, int F, int H, int init_random,
                                                             uint64_t seed, float scale) {
    __shared__ uint32_t used_s[kRwWaves][32];
    __shared__ uint32_t upre_s[kRwWaves][32];
    __shared__ int32_t feat_s[kRwWaves][kRwMaxF];
    __shared__ int32_t src_s[kRwWaves][kRwMaxF];
    __shared__ uint8_t mk_s[kRwWaves][kRwMaxF];
    __shared__ float row_s[kRwWaves][kRwMaxF];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int64_t k = (int64_t)blockIdx.x * kRwWaves + wv;
    if (k >= K) return;   // wave-uniform; this kernel has no workgroup barrier
    uint32_t *used = used_s[wv], *upre = upre_s[wv];
    int32_t *feat = feat_s[wv], *src = src_s[wv];
    uint8_t *mk = mk_s[wv];
    float *row = row_s[wv];
    const int64_t KF = K * F;

    // the group's slots, their marks (also as one 64-bit ballot per 64 slots), and the features it
    // keeps
    used[lane & 31] = 0u;
    constexpr int NPW = NPL;
    uint64_t pm[NPW];
    int n_pruned = 0;
#pragma unroll
    for (int w = 0; w < NPW; ++w) {
        const int j = lane + 64 * w;
        uint8_t m = 0;
        if (j < F) {
            feat[j] = idx[k * F + j];
            m = mask[k * F + j];
            mk[j] = m;
        }
        pm[w] = __builtin_amdgcn_ballot_w64(m != 0);
        n_pruned += __popcll(pm[w]);
    }
    if (n_pruned == 0) return;   // wave-uniform
    for (int j = lane; j < F; j += 64)
        if (!mk[j]) atomicOr(&used[feat[j] >> 5], 1u << (feat[j] & 31));

    // Draws, pruned slots in ascending order: the (r mod n_free)-th free feature, r the slot's
    // SplitMix64 value.  The d-th draw has n_free = H - (F - n_pruned) - d, so every draw's
    // r mod n_free is computed at once, on the lane of its slot; only the selection is sequential.
    // In 32-bit steps (n_free <= H <= 1024, so every product fits):
    //   r mod n = ((r_hi mod n) (2^32 mod n) + r_lo mod n) mod n.
    uint32_t tt[NPW];
    {
        int d0 = 0;   // pruned slots in earlier words
#pragma unroll
        for (int w = 0; w < NPW; ++w) {
            const int j = lane + 64 * w;
            tt[w] = 0u;
            if ((pm[w] >> lane) & 1u) {
                const int d = d0 + __popcll(pm[w] & ((1ull << lane) - 1ull));
                const uint64_t r = splitmix64_at(seed, (uint64_t)(k * F + j));
                const uint32_t nf = (uint32_t)(H - (F - n_pruned) - d);
                const uint32_t p32 = (0xFFFFFFFFu % nf + 1u) % nf;   // 2^32 mod nf
                tt[w] = ((uint32_t)(r >> 32) % nf * p32 % nf + (uint32_t)r % nf) % nf;
            }
            d0 += __popcll(pm[w]);
        }
    }
    // Lane w holds the free bits of bitmap word w (words past H have none) and the inclusive
    // prefix of the free counts, scanned once; a draw removes one bit, so the lane that held it
    // and every later prefix drop by one, with no further scan.
    const int nw = (H + 31) >> 5;
    uint32_t freew = 0u, valid = 0u;
    if (lane < nw) {
        const int lo = 32 * lane;
        valid = H - lo >= 32 ? 0xFFFFFFFFu : ((1u << (H - lo)) - 1u);
        freew = ~used[lane] & valid;
    }
    uint32_t c = __popc(freew), inc = c;
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t a = __shfl_up(inc, off, 64);
        if (lane >= off) inc += a;
    }
#pragma unroll
    for (int w = 0; w < NPW; ++w)
        for (uint64_t rem = pm[w]; rem != 0u; rem &= rem - 1u) {
            const int sl = (int)__builtin_ctzll(rem);
            const uint32_t t = __builtin_amdgcn_readlane(tt[w], sl);
            const uint32_t before = inc - c;
            const bool mine = before <= t && t < inc;
            // the holder's (t - before)-th free bit: a binary search on popcounts of halves
            uint32_t sel = mine ? t - before : 0u;
            int pos = 0;
#pragma unroll
            for (int half = 16; half > 0; half >>= 1) {
                const uint32_t cnt = __popc((freew >> pos) & ((1u << half) - 1u));
                if (sel >= cnt) {
                    sel -= cnt;
                    pos += half;
                }
            }
            const int holder = (int)__builtin_ctzll(__builtin_amdgcn_ballot_w64(mine));
            const int f = __builtin_amdgcn_readlane(32 * lane + pos, holder);
            if (lane == holder) {
                freew &= ~(1u << (f & 31));
                --c;
            }
            if (lane >= holder) --inc;
            if (lane == 0) feat[64 * w + sl] = f;
        }

    // new positions: the rank of each slot's feature among the row's features, from the final
    // bitmap (the features are distinct): used features in earlier words, plus the used bits of
    // its word below it
    {
        const uint32_t usedw = ~freew & valid;
        const uint32_t uc = __popc(usedw);
        uint32_t ui = uc;
        for (int off = 1; off < 64; off <<= 1) {
            const uint32_t a = __shfl_up(ui, off, 64);
            if (lane >= off) ui += a;
        }
        if (lane < nw) {
            used[lane] = usedw;
            upre[lane] = ui - uc;
        }
    }
    for (int j = lane; j < F; j += 64) {
        const int f = feat[j];
        const int p = (int)(upre[f >> 5] + __popc(used[f >> 5] & ((1u << (f & 31)) - 1u)));
        src[p] = j;
    }
    for (int p = lane; p < F; p += 64) idx[k * F + p] = feat[src[p]];

    // each label's weights (and velocity) follow their slots; pruned slots are reinitialised
    for (int g = 0; g < G; ++g) {
        const int64_t l = k * G + g;
        for (int j = lane; j < F; j += 64) row[j] = load_f32(W, l * F + j);
        for (int p = lane; p < F; p += 64) {
            const int j = src[p];
            float v = row[j];
            if (mk[j]) {
                v = 0.0f;
                if (init_random) {
                    const uint64_t n = splitmix64_at(seed, (uint64_t)(KF + l * F + j)) >> 40;
                    v = (float)((int32_t)(2 * n) - (1 << 24)) * scale;
                }
            }
            store_out(W, l * F + p, v);
        }
        if (mom) {
            for (int j = lane; j < F; j += 64) row[j] = mom[l * F + j];
            for (int p = lane; p < F; p += 64) mom[l * F + p] = mk[src[p]] ? 0.0f : row[src[p]];
        }
    }
}

}  // namespace

namespace haste {

// the regrowth addresses a group's weights (and velocity) with 32-bit offsets within its block
bool rewire_supported(const TailArgs &a) {
    return a.F_in <= kRwMaxF && a.F_s <= kMaxFs && a.G * a.F_in * 4 < ((int64_t)1 << 31);
}

static int64_t rw_blocks(const TailArgs &a) { return cdiv((a.L / a.G) * a.F_in, kRwBlock); }

size_t rewire_ws(const TailArgs &a) {
    const int64_t KF = (a.L / a.G) * a.F_in;
    return (size_t)round_up(KF * 4, 256) + (size_t)round_up(KF, 256) + (size_t)round_up(rw_blocks(a) * 4, 256) +
           256 * 4 + 256;
}

hipError_t rewire(const TailArgs &a, int32_t *idx, void *W, float *m, int64_t n_prune, int init_random, uint64_t seed,
                  void *ws, hipStream_t s) {
    const int64_t K = a.L / a.G, KF = K * a.F_in;
    char *p = static_cast<char *>(ws);
    uint32_t *keys = reinterpret_cast<uint32_t *>(p);
    p += round_up(KF * 4, 256);
    uint8_t *mask = reinterpret_cast<uint8_t *>(p);
    p += round_up(KF, 256);
    uint32_t *cnt = reinterpret_cast<uint32_t *>(p);
    p += round_up(rw_blocks(a) * 4, 256);
    uint32_t *hist = reinterpret_cast<uint32_t *>(p);
    RwState *st = reinterpret_cast<RwState *>(p + 256 * 4);
    const bool bf = a.dtype == HASTE_DTYPE_BF16;
    const dim3 g1((unsigned)cdiv(KF, 256));
    if (bf)
        hipLaunchKernelGGL((k_rw_scores<bf16_t>), g1, dim3(256), 0, s, (const bf16_t *)W, K, (int)a.G, (int)a.F_in, keys);
    else
        hipLaunchKernelGGL((k_rw_scores<float>), g1, dim3(256), 0, s, (const float *)W, K, (int)a.G, (int)a.F_in, keys);
    hipLaunchKernelGGL(k_rw_init, dim3(1), dim3(256), 0, s, hist, st, (uint64_t)(n_prune - 1));
    const int64_t hb = cdiv(KF, 1024) < 1024 ? (cdiv(KF, 1024) < 1 ? 1 : cdiv(KF, 1024)) : 1024;
    for (int shift = 24; shift >= 0; shift -= 8) {
        hipLaunchKernelGGL(k_rw_hist, dim3((unsigned)hb), dim3(256), 0, s, keys, KF, st, shift, hist);
        hipLaunchKernelGGL(k_rw_pick, dim3(1), dim3(256), 0, s, hist, st, shift);
    }
    const int64_t nb = rw_blocks(a);
    hipLaunchKernelGGL(k_rw_eqcount, dim3((unsigned)nb), dim3(256), 0, s, keys, KF, st, cnt);
    hipLaunchKernelGGL(k_rw_scan, dim3(1), dim3(kRwScanThreads), 0, s, cnt, nb);
    hipLaunchKernelGGL(k_rw_mark, dim3((unsigned)nb), dim3(256), 0, s, keys, KF, st, cnt, mask);
    const float scale = (float)(1.0 / sqrt((double)a.F_in)) * 5.9604644775390625e-08f;   // a 2^-24, exact
    const dim3 g2((unsigned)cdiv(K, kRwWaves));
    auto regrow = [&](auto tag, auto npl) {
        using T = decltype(tag);
        hipLaunchKernelGGL((k_rw_regrow<T, decltype(npl)::value>), g2, dim3(64 * kRwWaves), 0, s, idx, (T *)W, m,
                           mask, K, (int)a.G, (int)a.F_in, (int)a.F_s, init_random, seed, scale);
    };
    auto by_words = [&](auto tag) {
        if (a.F_in <= 64) regrow(tag, std::integral_constant<int, 1>{});
        else if (a.F_in <= 128) regrow(tag, std::integral_constant<int, 2>{});
        else regrow(tag, std::integral_constant<int, 4>{});
    };
    if (bf) by_words(bf16_t{});
    else by_words(float{});
    return hipGetLastError();
}

}  // namespace haste
