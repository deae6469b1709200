// Kernels of the batched search (paper Sec. 2.2.1: environments are scored by searching the
// player's action sequences; a node is a game state, an edge an action, and a state equal to
// one seen before keeps the node with the higher reward, then the shallower one).
//
// One level of a level-synchronous search over n children (parent i / A, action i % A):
//   gather    the frontier's packed rows are copied into the children batch, child i from
//             parent i / A, and the child's step counter starts at the parent's depth;
//   (step)    the children batch takes one step with the batch engines;
//   post      reward and depth are accumulated, the best (highest reward, earliest visit)
//             is kept with one 64-bit atomicMax, terminal children are counted, and every
//             other child hashes its packed map and finds its state's slot in the
//             open-addressing table (below): the slot's value becomes the max of
//             (reward, -depth) packed in 64 bits; a child that raised it stamps the slot with
//             this level's epoch;
//   claim     a child that took a fresh slot copies its map into the slot's map store and
//             marks the slot published; children whose value is the slot's value, in a slot
//             stamped this level, claim it with atomicMax(epoch, ~index): the lowest index
//             among the best wins;
//   flag      a child survives iff it holds its slot's claim; per-block survivor counts;
//   scan      exclusive prefix sum of the block counts (one workgroup);
//   place     survivors get their frontier position (block offset + in-block prefix);
//   copy      the next frontier's rows, reward and depth are gathered from the survivors.
// Table slots hold one state each and states are compared exactly: a slot's 64-bit key word
// is (32-bit tag of the map's hash) << 32 | owner, where the owner is kPending | child index
// while the slot was taken by a child of the running level (its map is that child's rows in
// the children batch) and kPublished once the map is in the slot's store entry.  A child
// probes from hash & mask: an empty slot is taken with one compare-and-swap of the whole
// word (tag and owner become visible together); a slot with its tag is the child's state iff
// the owner's map equals the child's map row for row; anything else probes the next slot.
// Equal hashes of different maps therefore never merge states; they only cost a comparison.
#include <algorithm>

#include "av_internal.h"

namespace av {
namespace {

constexpr uint32_t kMaxProbe = 4096;   // longest probe sequence before the table counts as full
constexpr uint32_t kPending = 0x80000000u;     // owner word: taken this level by child (low bits)
constexpr uint32_t kPublished = 0x40000000u;   // owner word: the map is in the slot's store entry

template <typename RowT>
__device__ inline uint64_t row_at(const void *base, size_t idx) {
    return uint64_t(static_cast<const RowT *>(base)[idx]);
}

// SplitMix64 finalizer (Steele, Lea, Flood, OOPSLA 2014): a bijective 64-bit mixer.
__device__ inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// Hash of environment i's map in a packed [C][n][H] buffer: one channel's H rows are H x
// sizeof(RowT) consecutive bytes; they are read as 64-bit little-endian words (the last one
// zero-padded) and the words of all channels, in channel order, are chained through the
// mixer: h = mix64(h ^ word).  0 is reserved for empty slots.
template <typename RowT>
__device__ inline uint64_t map_hash(const void *state, int i, int n, int C, int H) {
    uint64_t h = 0x9E3779B97F4A7C15ull;
    const int bytes = H * int(sizeof(RowT));
    for (int c = 0; c < C; ++c) {
        const RowT *blk = static_cast<const RowT *>(state) + (size_t(c) * n + i) * H;
        if (bytes % 16 == 0) {
            const uint4 *v = reinterpret_cast<const uint4 *>(blk);
            for (int k = 0; k < bytes / 16; ++k) {
                const uint4 q = v[k];
                h = mix64(h ^ (uint64_t(q.x) | (uint64_t(q.y) << 32)));
                h = mix64(h ^ (uint64_t(q.z) | (uint64_t(q.w) << 32)));
            }
        } else {
            constexpr int per = 8 / int(sizeof(RowT));
            for (int y0 = 0; y0 < H; y0 += per) {
                uint64_t word = 0;
                for (int k = 0; k < per && y0 + k < H; ++k)
                    word |= uint64_t(blk[y0 + k]) << (8 * int(sizeof(RowT)) * k);
                h = mix64(h ^ word);
            }
        }
    }
    return h ? h : 1;
}

// Copy environment blocks (one channel's H rows) 16 bytes per thread: destination block
// (c, i) of a [C][n][H] buffer comes from source block (c, from(i)) of a [C][nsrc][H] buffer,
// with from(i) = i / A (parents of the children) or src_of[i] (survivors).
// The destination is a [C][ndst][H] buffer written at blocks off .. off + n - 1.
__global__ void __launch_bounds__(256) copy16_kernel(const uint4 *src, int nsrc, uint4 *dst, int n,
                                                     int C, int chunks, int A,
                                                     const int32_t *src_of, int32_t *kid_t,
                                                     const int32_t *fdepth, int ndst, int off) {
    const size_t t = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (kid_t && t < size_t(n)) kid_t[t] = fdepth[t / A];
    if (t >= size_t(C) * n * chunks) return;
    const int k = int(t % chunks);
    const size_t ci = t / chunks;
    const int i = int(ci % n), c = int(ci / n);
    const int from = src_of ? src_of[i] : i / A;
    dst[(size_t(c) * ndst + off + i) * chunks + k] = src[(size_t(c) * nsrc + from) * chunks + k];
}

__device__ inline uint64_t pack_value(int32_t reward, int32_t depth) {
    return (uint64_t(uint32_t(reward) ^ 0x80000000u) << 32) | uint64_t(0xFFFFFFFFu - uint32_t(depth));
}

__device__ inline uint32_t hash_tag(uint64_t h) { return uint32_t(h >> 32) ^ uint32_t(h); }

// Do environment i of the packed [C][n][H] buffer `kids` and the map `other` hold the same
// rows?  `other` is environment j of the same buffer (j >= 0) or a store entry ([C][H] rows).
template <typename RowT>
__device__ inline bool same_map(const void *kids, int n, int i, int j, const void *other, int C,
                                int H) {
    const RowT *a = static_cast<const RowT *>(kids);
    const RowT *b = j >= 0 ? a : static_cast<const RowT *>(other);
    if ((H * sizeof(RowT)) % 16 == 0) {
        // a channel's rows are whole 16-byte words at 16-byte aligned offsets (buffers from
        // hipMalloc, blocks of H rows): compared 16 bytes at a time
        const int q = int(H * sizeof(RowT) / 16);
        for (int c = 0; c < C; ++c) {
            const uint4 *ra = reinterpret_cast<const uint4 *>(a + (size_t(c) * n + i) * H);
            const uint4 *rb = reinterpret_cast<const uint4 *>(
                j >= 0 ? b + (size_t(c) * n + j) * H : b + size_t(c) * H);
            for (int k = 0; k < q; ++k) {
                const uint4 x = ra[k], z = rb[k];
                if ((x.x ^ z.x) | (x.y ^ z.y) | (x.z ^ z.z) | (x.w ^ z.w)) return false;
            }
        }
        return true;
    }
    for (int c = 0; c < C; ++c) {
        const RowT *ra = a + (size_t(c) * n + i) * H;
        const RowT *rb = j >= 0 ? b + (size_t(c) * n + j) * H : b + size_t(c) * H;
        for (int y = 0; y < H; ++y)
            if (ra[y] != rb[y]) return false;
    }
    return true;
}

// The slot of child i's state (hash h): an equal map found on its probe path, or the first
// empty slot, taken for child i (*fresh = true).  -1 when kMaxProbe slots all hold other
// states.
template <typename RowT>
__device__ inline int64_t probe_exact(const SearchArgs &a, const void *kids, int i, uint64_t h,
                                      bool *fresh) {
    const uint32_t tag = hash_tag(h);
    const unsigned long long mine =
        (static_cast<unsigned long long>(tag) << 32) | (kPending | uint32_t(i));
    const size_t sbytes = size_t(a.C) * a.H * sizeof(RowT);
    uint64_t s = h & a.mask;
    *fresh = false;
    for (uint32_t k = 0; k < kMaxProbe; ++k) {
        const uint64_t prev =
            atomicCAS(reinterpret_cast<unsigned long long *>(&a.keys[s]), 0ull, mine);
        if (prev == 0) {
            *fresh = true;
            return int64_t(s);
        }
        if (uint32_t(prev >> 32) == tag) {
            const uint32_t own = uint32_t(prev);
            const bool eq = (own & kPending)
                                ? same_map<RowT>(kids, a.n, i, int(own & ~kPending), nullptr,
                                                 a.C, a.H)
                                : same_map<RowT>(kids, a.n, i, -1,
                                                 static_cast<const char *>(a.store) + s * sbytes,
                                                 a.C, a.H);
            if (eq) return int64_t(s);
        }
        s = (s + 1) & a.mask;
    }
    return -1;
}

template <typename RowT>
__global__ void __launch_bounds__(256) gather_kernel(const void *front, int nf, const int32_t *fdepth,
                                                     void *kids, int32_t *kid_t, int n, int A,
                                                     int C, int H) {
    const size_t r = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
    const size_t rows = size_t(C) * n * H;
    if (r < size_t(n)) kid_t[r] = fdepth[r / A];
    if (r >= rows) return;
    const int y = int(r % H);
    const size_t ci = r / H;
    const int i = int(ci % n), c = int(ci / n);
    const int p = i / A;
    static_cast<RowT *>(kids)[r] = static_cast<const RowT *>(front)[(size_t(c) * nf + p) * H + y];
}

template <typename RowT>
__global__ void __launch_bounds__(256) post_kernel(SearchArgs a, const void *kids, const float *rew,
                                                   const uint8_t *done) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= a.n) return;
    const int p = i / a.A;
    const int32_t reward = a.front_reward[p] + int32_t(rew[i]);
    const int32_t depth = a.front_depth[p] + 1;
    const uint64_t visit = a.visited + 1 + uint64_t(i);
    atomicMax(reinterpret_cast<unsigned long long *>(a.best),
              static_cast<unsigned long long>((uint64_t(uint32_t(reward) ^ 0x80000000u) << 32) |
                                              (0xFFFFFFFFull - visit)));
    a.kid_reward[i] = reward;
    a.kid_depth[i] = depth;
    a.slot[i] = -1;
    if (done[i]) {
        atomicAdd(&a.counts[0], 1u);
        return;
    }
    const uint64_t h = map_hash<RowT>(kids, i, a.n, a.C, a.H) & a.hash_mask;
    bool fresh;
    const int64_t s = probe_exact<RowT>(a, kids, i, h, &fresh);
    if (s < 0) {
        atomicOr(&a.counts[1], 1u);
        return;
    }
    const uint64_t v = pack_value(reward, depth);
    const uint64_t old = atomicMax(reinterpret_cast<unsigned long long *>(&a.vals[s]),
                                   static_cast<unsigned long long>(v));
    if (old < v) a.epoch[s] = a.cur_epoch;
    a.slot[i] = s;
    a.kid_val[i] = v;
}

template <typename RowT>
__global__ void __launch_bounds__(256) claim_kernel(SearchArgs a, const void *kids) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= a.n) return;
    const int64_t s = a.slot[i];
    if (s < 0) return;
    // publish a slot this child took: its map into the store, then the owner word (in this
    // kernel the store is not read, and the other children of the slot read the key word
    // only to see that it is not theirs; the next level sees both)
    const uint64_t key = a.keys[s];
    if (uint32_t(key) == (kPending | uint32_t(i))) {
        RowT *dst = reinterpret_cast<RowT *>(static_cast<char *>(a.store) +
                                             size_t(s) * a.C * a.H * sizeof(RowT));
        const RowT *src = static_cast<const RowT *>(kids);
        if ((a.H * sizeof(RowT)) % 16 == 0) {          // 16 bytes at a time (see same_map)
            const int q = int(a.H * sizeof(RowT) / 16);
            for (int c = 0; c < a.C; ++c) {
                const uint4 *from = reinterpret_cast<const uint4 *>(src + (size_t(c) * a.n + i) * a.H);
                uint4 *to = reinterpret_cast<uint4 *>(dst + size_t(c) * a.H);
                for (int k = 0; k < q; ++k) to[k] = from[k];
            }
        } else {
            for (int c = 0; c < a.C; ++c)
                for (int y = 0; y < a.H; ++y) dst[c * a.H + y] = src[(size_t(c) * a.n + i) * a.H + y];
        }
        a.keys[s] = (key & 0xFFFFFFFF00000000ull) | kPublished;
    }
    if (a.vals[s] == a.kid_val[i] && a.epoch[s] == a.cur_epoch)
        atomicMax(reinterpret_cast<unsigned long long *>(&a.claim[s]),
                  static_cast<unsigned long long>((uint64_t(a.cur_epoch) << 32) |
                                                  (0xFFFFFFFFu - uint32_t(i))));
}

__device__ inline bool survives(const SearchArgs &a, int i) {
    const int64_t s = a.slot[i];
    return s >= 0 && a.vals[s] == a.kid_val[i] && a.epoch[s] == a.cur_epoch &&
           a.claim[s] == ((uint64_t(a.cur_epoch) << 32) | (0xFFFFFFFFu - uint32_t(i)));
}

// In-block exclusive prefix of 0/1 flags (256 threads, four waves); returns the block total.
__device__ inline int block_prefix(int flag, int *sums, int &prefix) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint64_t ballot = __ballot(flag);
    const int in_wave = __popcll(ballot & ((lane ? (~0ull >> (64 - lane)) : 0ull)));
    if (lane == 0) sums[wave] = __popcll(ballot);
    __syncthreads();
    int before = 0, total = 0;
    for (int w = 0; w < 4; ++w) {
        if (w < wave) before += sums[w];
        total += sums[w];
    }
    prefix = before + in_wave;
    return total;
}

__global__ void __launch_bounds__(256) flag_kernel(SearchArgs a) {
    __shared__ int sums[4];
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    const int flag = i < a.n && survives(a, i);
    int prefix;
    const int total = block_prefix(flag, sums, prefix);
    if (threadIdx.x == 0) a.block_count[blockIdx.x] = total;
}

// Exclusive scan of the per-block counts; one workgroup of 256 threads; also the total.
__global__ void __launch_bounds__(256) scan_kernel(int32_t *block_count, int nb, uint32_t *total) {
    __shared__ int part[256];
    const int t = threadIdx.x;
    const int per = (nb + 255) / 256;
    const int lo = t * per, hi = lo + per < nb ? lo + per : nb;
    int sum = 0;
    for (int k = lo; k < hi; ++k) sum += block_count[k];
    part[t] = sum;
    __syncthreads();
    if (t == 0) {
        int run = 0;
        for (int k = 0; k < 256; ++k) {
            const int v = part[k];
            part[k] = run;
            run += v;
        }
        *total = uint32_t(run);
    }
    __syncthreads();
    int run = part[t];
    for (int k = lo; k < hi; ++k) {
        const int v = block_count[k];
        block_count[k] = run;
        run += v;
    }
}

__global__ void __launch_bounds__(256) place_kernel(SearchArgs a, int cap) {
    __shared__ int sums[4];
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    const int flag = i < a.n && survives(a, i);
    int prefix;
    block_prefix(flag, sums, prefix);
    if (!flag) return;
    const int pos = a.block_count[blockIdx.x] + prefix;
    if (pos >= cap) return;
    a.src_of[pos] = i;
    a.next_reward[pos] = a.kid_reward[i];
    a.next_depth[pos] = a.kid_depth[i];
}

// Rows of blocks src_of[q] of a [C][n][H] buffer into blocks off + q of a [C][ndst][H] one.
template <typename RowT>
__global__ void __launch_bounds__(256) copy_kernel(const void *kids, int n, void *next, int nn,
                                                   const int32_t *src_of, int C, int H, int ndst,
                                                   int off) {
    const size_t r = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (r >= size_t(C) * nn * H) return;
    const int y = int(r % H);
    const size_t cq = r / H;
    const int q = int(cq % nn), c = int(cq / nn);
    static_cast<RowT *>(next)[(size_t(c) * ndst + off + q) * H + y] =
        static_cast<const RowT *>(kids)[(size_t(c) * n + src_of[q]) * H + y];
}

template <typename RowT>
__global__ void root_kernel(SearchArgs a, const void *front) {
    if (blockIdx.x != 0 || threadIdx.x != 0) return;
    // the table is empty: the root takes its home slot, published at once
    const uint64_t h = map_hash<RowT>(front, 0, 1, a.C, a.H) & a.hash_mask;
    const uint64_t s = h & a.mask;
    RowT *dst = reinterpret_cast<RowT *>(static_cast<char *>(a.store) +
                                         size_t(s) * a.C * a.H * sizeof(RowT));
    for (int r = 0; r < a.C * a.H; ++r) dst[r] = static_cast<const RowT *>(front)[r];
    a.keys[s] = (uint64_t(hash_tag(h)) << 32) | kPublished;
    a.vals[s] = pack_value(0, 0);
    *a.best = (uint64_t(0x80000000u) << 32) | 0xFFFFFFFFull;
    if (a.root_slot) *a.root_slot = s;
}

// ---------------------------------------------------------------------------------------
// Batched best-first (av_search_config.best_first_k > 0).  Nodes live in a pool ([C][P][H]
// rows plus reward, depth, packed (reward, -depth) value and table slot per node id); the
// open list holds (value, id) pairs sorted by value descending, ties by id ascending.  An
// iteration pops its first k entries, keeps those whose value is still their slot's value
// (the others were beaten by a later copy of their state), expands them in id order with the
// level kernels above, appends the survivors to the pool with the next ids, sorts them, and
// merges them into the rest of the open list.

// In-block exclusive prefix of 0/1 flags for any multiple of 64 threads (up to 1024).
__device__ inline int block_prefix_any(int flag, int *sums, int &prefix) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const uint64_t ballot = __ballot(flag);
    const int in_wave = __popcll(ballot & ((lane ? (~0ull >> (64 - lane)) : 0ull)));
    if (lane == 0) sums[wave] = __popcll(ballot);
    __syncthreads();
    int before = 0, total = 0;
    for (int w = 0; w < nw; ++w) {
        if (w < wave) before += sums[w];
        total += sums[w];
    }
    prefix = before + in_wave;
    return total;
}

// Pop: the first kp open ids, sorted ascending (bitonic, 512 slots), those still alive
// compacted into parents[]; *n_par = their number.  One workgroup of 512 threads.
__global__ void __launch_bounds__(512) bf_pop_kernel(const uint32_t *open_ids, int kp,
                                                     const int64_t *pool_slot,
                                                     const uint64_t *pool_val,
                                                     const uint64_t *vals, int32_t *parents,
                                                     uint32_t *n_par, uint32_t *counts) {
    __shared__ uint32_t ids[512];
    if (threadIdx.x < 3) counts[threadIdx.x] = 0u;   // the level's counters, for what follows
    __shared__ int sums[8];
    const int t = threadIdx.x;
    ids[t] = t < kp ? open_ids[t] : 0xFFFFFFFFu;
    __syncthreads();
    // a bitonic network over the first P = next power of two >= kp entries (the rest hold the
    // largest id and stay in place)
    const int P = kp <= 1 ? 1 : 1 << (32 - __builtin_clz(uint32_t(kp - 1)));
    for (int k = 2; k <= P; k <<= 1)
        for (int j = k >> 1; j > 0; j >>= 1) {
            const int o = t ^ j;
            if (t < P && o > t) {
                const uint32_t a = ids[t], b = ids[o];
                const bool up = (t & k) == 0;
                if ((a > b) == up) {
                    ids[t] = b;
                    ids[o] = a;
                }
            }
            __syncthreads();
        }
    const uint32_t id = ids[t];
    const int alive = id != 0xFFFFFFFFu && vals[pool_slot[id]] == pool_val[id];
    int prefix;
    const int total = block_prefix_any(alive, sums, prefix);
    if (alive) parents[prefix] = int32_t(id);
    if (t == 0) *n_par = uint32_t(total);
}

__global__ void __launch_bounds__(256) bf_gather_meta(const int32_t *parents, int np,
                                                      const int32_t *pool_reward,
                                                      const int32_t *pool_depth,
                                                      int32_t *front_reward, int32_t *front_depth) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= np) return;
    front_reward[i] = pool_reward[parents[i]];
    front_depth[i] = pool_depth[parents[i]];
}

// New nodes pool_n + q (q < nn) from survivor children src_of[q]: value and slot, and the
// (value, id) pairs to sort.  Reward and depth were written by place_kernel.
__global__ void __launch_bounds__(256) bf_append_meta(const int32_t *src_of, int nn, int pool_n,
                                                      const uint64_t *kid_val, const int64_t *slot,
                                                      uint64_t *pool_val, int64_t *pool_slot,
                                                      uint64_t *new_keys, uint32_t *new_ids) {
    const int q = blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= nn) return;
    const int i = src_of[q];
    pool_val[pool_n + q] = kid_val[i];
    pool_slot[pool_n + q] = slot[i];
    new_keys[q] = kid_val[i];
    new_ids[q] = uint32_t(pool_n + q);
}

// Sort nn <= 4096 (value, id) pairs: value descending, id ascending (bitonic in LDS).
__global__ void __launch_bounds__(1024) bf_sort_kernel(uint64_t *keys, uint32_t *ids, int nn) {
    __shared__ uint64_t k_[4096];
    __shared__ uint32_t i_[4096];
    int P = 1;
    while (P < nn) P <<= 1;
    for (int t = threadIdx.x; t < P; t += blockDim.x) {
        k_[t] = t < nn ? keys[t] : 0ull;
        i_[t] = t < nn ? ids[t] : 0xFFFFFFFFu;
    }
    __syncthreads();
    for (int k = 2; k <= P; k <<= 1)
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int t = threadIdx.x; t < P; t += blockDim.x) {
                const int o = t ^ j;
                if (o > t) {
                    // "a before b": larger value, or equal value and smaller id
                    const bool b_first = k_[o] > k_[t] || (k_[o] == k_[t] && i_[o] < i_[t]);
                    const bool up = (t & k) == 0;
                    if (b_first == up) {
                        const uint64_t kk = k_[t];
                        k_[t] = k_[o];
                        k_[o] = kk;
                        const uint32_t ii = i_[t];
                        i_[t] = i_[o];
                        i_[o] = ii;
                    }
                }
            }
            __syncthreads();
        }
    for (int t = threadIdx.x; t < nn; t += blockDim.x) {
        keys[t] = k_[t];
        ids[t] = i_[t];
    }
}

// Merge the old open list (m pairs) with the sorted new pairs (nn) into out: old entries
// come before new ones of equal value (their ids are smaller).
__global__ void __launch_bounds__(256) bf_merge_kernel(const uint64_t *ok, const uint32_t *oi, int m,
                                                       const uint64_t *nk, const uint32_t *ni, int nn,
                                                       uint64_t *outk, uint32_t *outi) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t < m) {
        const uint64_t key = ok[t];
        int lo = 0, hi = nn;                       // new entries with a larger value
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (nk[mid] > key) lo = mid + 1; else hi = mid;
        }
        outk[t + lo] = key;
        outi[t + lo] = oi[t];
    } else if (t < m + nn) {
        const int q = t - m;
        const uint64_t key = nk[q];
        int lo = 0, hi = m;                        // old entries with a value >= this one
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (ok[mid] >= key) lo = mid + 1; else hi = mid;
        }
        outk[q + lo] = key;
        outi[q + lo] = ni[q];
    }
}

template <typename RowT>
__global__ void __launch_bounds__(256) bf_unpack_kernel(const void *pool, int pcap,
                                                        const uint32_t *ids, int n, int C, int H,
                                                        int W, uint8_t *maps) {
    const size_t r = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (r >= size_t(n) * C * H) return;
    const int y = int(r % H);
    const size_t qc = r / H;
    const int c = int(qc % C), q = int(qc / C);
    const uint64_t v = uint64_t(static_cast<const RowT *>(pool)[(size_t(c) * pcap + ids[q]) * H + y]);
    uint8_t *o = maps + r * W;
    for (int x = 0; x < W; ++x) o[x] = uint8_t((v >> x) & 1u);
}

__global__ void __launch_bounds__(256) bf_open_meta(const uint32_t *ids, int n,
                                                    const int32_t *pool_reward,
                                                    const int32_t *pool_depth, int32_t *reward,
                                                    int32_t *depth) {
    const int q = blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= n) return;
    if (reward) reward[q] = pool_reward[ids[q]];
    if (depth) depth[q] = pool_depth[ids[q]];
}

unsigned blocks_for(size_t threads) { return unsigned((threads + 255) / 256); }

template <typename RowT>
hipError_t level_impl(const SearchArgs &a, const void *front, int nf, void *kids, int32_t *kid_t,
                      hipStream_t s, int phase, int nn) {
    const int block_bytes = a.H * int(sizeof(RowT));
    const bool by16 = block_bytes % 16 == 0;
    const int chunks = block_bytes / 16;
    if (phase == 0) {
        if (by16) {
            const size_t threads = std::max(size_t(a.C) * a.n * chunks, size_t(a.n));
            hipLaunchKernelGGL(copy16_kernel, dim3(blocks_for(threads)), dim3(256), 0, s,
                               static_cast<const uint4 *>(front), nf, static_cast<uint4 *>(kids),
                               a.n, a.C, chunks, a.A, static_cast<const int32_t *>(nullptr),
                               kid_t, a.front_depth, a.n, 0);
        } else {
            const size_t rows = std::max(size_t(a.C) * a.n * a.H, size_t(a.n));
            hipLaunchKernelGGL(gather_kernel<RowT>, dim3(blocks_for(rows)), dim3(256), 0, s, front,
                               nf, a.front_depth, kids, kid_t, a.n, a.A, a.C, a.H);
        }
    } else if (phase == 1) {
        const unsigned nb = blocks_for(size_t(a.n));
        hipLaunchKernelGGL(post_kernel<RowT>, dim3(nb), dim3(256), 0, s, a, kids, a.rew, a.done);
        hipLaunchKernelGGL(claim_kernel<RowT>, dim3(nb), dim3(256), 0, s, a, kids);
        hipLaunchKernelGGL(flag_kernel, dim3(nb), dim3(256), 0, s, a);
        hipLaunchKernelGGL(scan_kernel, dim3(1), dim3(256), 0, s, a.block_count, int(nb),
                           &a.counts[2]);
        hipLaunchKernelGGL(place_kernel, dim3(nb), dim3(256), 0, s, a, a.cap);
    } else if (phase == 2) {
        if (nn > 0 && by16)
            hipLaunchKernelGGL(copy16_kernel, dim3(blocks_for(size_t(a.C) * nn * chunks)), dim3(256),
                               0, s, static_cast<const uint4 *>(kids), a.n,
                               static_cast<uint4 *>(a.next), nn, a.C, chunks, 1,
                               static_cast<const int32_t *>(a.src_of),
                               static_cast<int32_t *>(nullptr),
                               static_cast<const int32_t *>(nullptr), a.next_n, a.next_off);
        else if (nn > 0)
            hipLaunchKernelGGL(copy_kernel<RowT>, dim3(blocks_for(size_t(a.C) * nn * a.H)), dim3(256),
                               0, s, kids, a.n, a.next, nn, a.src_of, a.C, a.H, a.next_n,
                               a.next_off);
    } else {
        hipLaunchKernelGGL(root_kernel<RowT>, dim3(1), dim3(64), 0, s, a, front);
    }
    return hipGetLastError();
}

template <typename RowT>
hipError_t copy_rows(const void *src, int nsrc, const int32_t *src_of, void *dst, int ndst,
                     int off, int n, int C, int H, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const int block_bytes = H * int(sizeof(RowT));
    if (block_bytes % 16 == 0) {
        const int chunks = block_bytes / 16;
        hipLaunchKernelGGL(copy16_kernel, dim3(blocks_for(size_t(C) * n * chunks)), dim3(256), 0, s,
                           static_cast<const uint4 *>(src), nsrc, static_cast<uint4 *>(dst), n, C,
                           chunks, 1, src_of, static_cast<int32_t *>(nullptr),
                           static_cast<const int32_t *>(nullptr), ndst, off);
    } else {
        hipLaunchKernelGGL(copy_kernel<RowT>, dim3(blocks_for(size_t(C) * n * H)), dim3(256), 0, s,
                           src, nsrc, dst, n, src_of, C, H, ndst, off);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_copy_rows(int row_bytes, const void *src, int nsrc, const int32_t *src_of,
                            void *dst, int ndst, int off, int n, int C, int H, hipStream_t s) {
    if (row_bytes == 2) return copy_rows<uint16_t>(src, nsrc, src_of, dst, ndst, off, n, C, H, s);
    if (row_bytes == 4) return copy_rows<uint32_t>(src, nsrc, src_of, dst, ndst, off, n, C, H, s);
    return copy_rows<uint64_t>(src, nsrc, src_of, dst, ndst, off, n, C, H, s);
}

hipError_t launch_bf_pop(const uint32_t *open_ids, int kp, const int64_t *pool_slot,
                         const uint64_t *pool_val, const uint64_t *vals, int32_t *parents,
                         uint32_t *n_par, uint32_t *counts, hipStream_t s) {
    hipLaunchKernelGGL(bf_pop_kernel, dim3(1), dim3(512), 0, s, open_ids, kp, pool_slot, pool_val,
                       vals, parents, n_par, counts);
    return hipGetLastError();
}

hipError_t launch_bf_gather_meta(const int32_t *parents, int np, const int32_t *pool_reward,
                                 const int32_t *pool_depth, int32_t *front_reward,
                                 int32_t *front_depth, hipStream_t s) {
    if (np <= 0) return hipSuccess;
    hipLaunchKernelGGL(bf_gather_meta, dim3(blocks_for(size_t(np))), dim3(256), 0, s, parents, np,
                       pool_reward, pool_depth, front_reward, front_depth);
    return hipGetLastError();
}

hipError_t launch_bf_append(const int32_t *src_of, int nn, int pool_n, const uint64_t *kid_val,
                            const int64_t *slot, uint64_t *pool_val, int64_t *pool_slot,
                            uint64_t *new_keys, uint32_t *new_ids, hipStream_t s) {
    if (nn <= 0) return hipSuccess;
    hipLaunchKernelGGL(bf_append_meta, dim3(blocks_for(size_t(nn))), dim3(256), 0, s, src_of, nn,
                       pool_n, kid_val, slot, pool_val, pool_slot, new_keys, new_ids);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(bf_sort_kernel, dim3(1), dim3(1024), 0, s, new_keys, new_ids, nn);
    return hipGetLastError();
}

hipError_t launch_bf_merge(const uint64_t *ok, const uint32_t *oi, int m, const uint64_t *nk,
                           const uint32_t *ni, int nn, uint64_t *outk, uint32_t *outi,
                           hipStream_t s) {
    if (m + nn <= 0) return hipSuccess;
    hipLaunchKernelGGL(bf_merge_kernel, dim3(blocks_for(size_t(m) + nn)), dim3(256), 0, s, ok, oi, m,
                       nk, ni, nn, outk, outi);
    return hipGetLastError();
}

hipError_t launch_bf_open(int row_bytes, const void *pool, int pcap, const uint32_t *ids, int n,
                          int C, int H, int W, uint8_t *maps, const int32_t *pool_reward,
                          const int32_t *pool_depth, int32_t *reward, int32_t *depth,
                          hipStream_t s) {
    if (n <= 0) return hipSuccess;
    if (maps) {
        const unsigned nb = blocks_for(size_t(n) * C * H);
        if (row_bytes == 2)
            hipLaunchKernelGGL(bf_unpack_kernel<uint16_t>, dim3(nb), dim3(256), 0, s, pool, pcap, ids,
                               n, C, H, W, maps);
        else if (row_bytes == 4)
            hipLaunchKernelGGL(bf_unpack_kernel<uint32_t>, dim3(nb), dim3(256), 0, s, pool, pcap, ids,
                               n, C, H, W, maps);
        else
            hipLaunchKernelGGL(bf_unpack_kernel<uint64_t>, dim3(nb), dim3(256), 0, s, pool, pcap, ids,
                               n, C, H, W, maps);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (reward || depth)
        hipLaunchKernelGGL(bf_open_meta, dim3(blocks_for(size_t(n))), dim3(256), 0, s, ids, n,
                           pool_reward, pool_depth, reward, depth);
    return hipGetLastError();
}

hipError_t launch_search_phase(const SearchArgs &a, int row_bytes, const void *front, int nf,
                               void *kids, int32_t *kid_t, hipStream_t s, int phase, int nn) {
    if (row_bytes == 2) return level_impl<uint16_t>(a, front, nf, kids, kid_t, s, phase, nn);
    if (row_bytes == 4) return level_impl<uint32_t>(a, front, nf, kids, kid_t, s, phase, nn);
    return level_impl<uint64_t>(a, front, nf, kids, kid_t, s, phase, nn);
}

}  // namespace av
