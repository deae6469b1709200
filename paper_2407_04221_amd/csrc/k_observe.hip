// Observation kernel: the player-centred window of every environment's current map
// (paper Sec. 2.2.2: a local patch of tiles around the player's position; Table 1 uses
// windows of 5, 10, 20 and 31 cells).
//
// 16, 32 or 64 lanes per environment (more for larger outputs), 256 lanes to a workgroup.
// The environment's packed rows are staged in LDS; the first player cell in row-major order
// is found with an LDS atomicMin over rows (then the row's lowest set bit).  Where it fits in
// LDS, the window is then laid out as a bit string (bit o for output byte o), one shift and
// mask of a staged row per window row OR-ed in with LDS atomics; otherwise each chunk's cells
// are gathered from the staged rows directly, one shift per window row the chunk touches.
// The C x w x w output bytes are written in 16-byte chunks on the global 16-byte grid, one
// chunk per thread and pass, as a 16-bit mask whose every 4 bits are spread into 4 bytes
// with one multiply (bit i of v & 15 lands in byte i of (v & 15) * 0x204081); the bytes
// before the first and after the last full chunk are written one by one.  Window cell
// (wy, wx) shows map cell (py - w/2 + wy, px - w/2 + wx); cells off the map, and the whole
// window of a map without a player, are 0 (packed rows hold no bits at x >= W).
#include "av_internal.h"

namespace av {
namespace {

__device__ inline uint64_t load_row(const void *base, size_t idx, int row_bytes) {
    if (row_bytes == 2) return static_cast<const uint16_t *>(base)[idx];
    if (row_bytes == 4) return static_cast<const uint32_t *>(base)[idx];
    return static_cast<const uint64_t *>(base)[idx];
}

__device__ inline int lowbit(uint64_t v) { return __ffsll(static_cast<unsigned long long>(v)) - 1; }

// Map bits x0 .. x0 + 63 of a row as the low bits of the result (0 outside the row).
__device__ inline uint64_t row_from(uint64_t row, int x0) {
    if (x0 >= 64 || x0 <= -64) return 0ull;
    return x0 >= 0 ? row >> x0 : row << -x0;
}

// Position of output byte o of one environment: channel c, window row wy, column wx.
// (One environment's output is at most 31 x 255 x 255 bytes, so offsets fit 32 bits.)
struct WinPos {
    int c, wy, wx;
};
__device__ inline WinPos win_pos(uint32_t o, int w) {
    const uint32_t ww = uint32_t(w) * uint32_t(w);
    const int c = int(o / ww);
    const uint32_t rem = o - uint32_t(c) * ww;
    const int wy = int(rem / uint32_t(w));
    return {c, wy, int(rem - uint32_t(wy) * uint32_t(w))};
}

// The window cells of n output bytes (n <= 16) from position (c, wy, wx) on, as a mask, bit k
// for the k-th byte.  rows: the environment's staged planes [C][H]; (y0, x0) the window's
// top-left map cell.
__device__ inline uint32_t window_bits(const uint64_t *rows, int H, int w, bool has, int y0,
                                       int x0, WinPos p, int n) {
    int c = p.c, wy = p.wy, wx = p.wx;
    uint32_t m = 0;
    for (int k = 0; k < n;) {
        const int len = min(n - k, w - wx);
        const int y = y0 + wy;
        const uint64_t row = (has && y >= 0 && y < H) ? rows[size_t(c) * H + y] : 0ull;
        m |= uint32_t(row_from(row, x0 + wx) & ((1ull << len) - 1ull)) << k;
        k += len;
        wx += len;
        if (wx == w) {
            wx = 0;
            if (++wy == w) {
                wy = 0;
                ++c;
            }
        }
    }
    return m;
}

// Four bytes 0/1 from the low 4 bits of v (bit i -> byte i).
__device__ inline uint32_t spread4(uint32_t v) { return ((v & 15u) * 0x204081u) & 0x01010101u; }

// The window's map bits for window row r (channel r / w, row r % w) OR-ed into the bit string
// wb at bits r w .. r w + w - 1 (bit o of wb is output byte o).  Only map columns inside the
// window contribute, so every bit set lies inside the row's own w bits.
__device__ inline void window_row_to_bits(const uint64_t *rows, int H, int w, int y0, int x0,
                                          int r, uint32_t *wb) {
    const int c = r / w, y = y0 + (r - c * w);
    if (y < 0 || y >= H) return;
    const int sh = x0 > 0 ? x0 : 0;     // map columns left of the window
    const int off = x0 < 0 ? -x0 : 0;   // window columns left of the map
    const int len = w - off;            // window columns from the map's first column on
    if (len <= 0 || sh >= 64) return;
    uint64_t bits = rows[size_t(c) * H + y] >> sh;
    if (len < 64) bits &= (1ull << len) - 1ull;
    if (!bits) return;
    const uint32_t pos = uint32_t(r) * uint32_t(w) + uint32_t(off);
    const uint32_t wi = pos >> 5, bi = pos & 31u;
    atomicOr(&wb[wi], uint32_t(bits << bi));
    const uint32_t mid = bi ? uint32_t(bits >> (32u - bi)) : uint32_t(bits >> 32);
    const uint32_t hi = bi ? uint32_t(bits >> (64u - bi)) : 0u;
    if (mid) atomicOr(&wb[wi + 1], mid);
    if (hi) atomicOr(&wb[wi + 2], hi);
}

// T threads per environment, 256 / T environments per workgroup, `region` LDS bytes each: the
// staged rows and the player row at the front (`base` bytes), then, with kStream, the window
// as a bit string of `sw` words (bit o = output byte o, two words of zero padding).
template <int T, bool kStream>
__global__ void __launch_bounds__(256) observe_env(const void *state, int B, int C, int H, int W,
                                                   int row_bytes, int w, uint8_t *dst, int region,
                                                   int base, int sw) {
    extern __shared__ __align__(16) unsigned char lds[];
    constexpr int G = 256 / T;
    const int tid = threadIdx.x % T, slot = threadIdx.x / T;
    const int b = blockIdx.x * G + slot;
    const bool live = b < B;
    uint64_t *rows = reinterpret_cast<uint64_t *>(lds + size_t(slot) * region);   // [C][H]
    int *first = reinterpret_cast<int *>(rows + size_t(C) * H);
    uint32_t *wb = reinterpret_cast<uint32_t *>(lds + size_t(slot) * region + base);   // [sw]
    if (tid == 0) *first = H;
    if (live) {
        for (int r = tid; r < C * H; r += T) {
            const int c = r / H, y = r - c * H;
            rows[r] = load_row(state, (size_t(c) * B + b) * H + y, row_bytes);
        }
        if (kStream)
            for (int i = tid; i < sw; i += T) wb[i] = 0u;
    }
    __syncthreads();
    if (live)
        for (int y = tid; y < H; y += T)
            if (rows[size_t(kChPlayer) * H + y]) atomicMin(first, y);
    __syncthreads();
    const int py = *first;
    const bool has = live && py < H;
    const int px = has ? lowbit(rows[size_t(kChPlayer) * H + py]) : 0;
    const int y0 = py - w / 2, x0 = px - w / 2;
    (void)W;
    if (kStream) {
        if (has)
            for (int r = tid; r < C * w; r += T) window_row_to_bits(rows, H, w, y0, x0, r, wb);
        __syncthreads();
    }
    if (!live) return;

    const uint32_t per = uint32_t(C) * uint32_t(w) * uint32_t(w);
    uint8_t *const out = dst + size_t(b) * per;
    const uint32_t head = uint32_t(16 - (reinterpret_cast<uintptr_t>(out) & 15)) & 15u;
    const uint32_t h = head < per ? head : per;
    const uint32_t chunks = (per - h) / 16;
    if (kStream) {
        for (uint32_t k = tid; k < chunks; k += T) {
            const uint32_t o = h + 16 * k, i = o >> 5;
            const uint64_t two = uint64_t(wb[i]) | (uint64_t(wb[i + 1]) << 32);
            const uint32_t m = uint32_t(two >> (o & 31u));
            *reinterpret_cast<uint4 *>(out + o) =
                make_uint4(spread4(m), spread4(m >> 4), spread4(m >> 8), spread4(m >> 12));
        }
    } else {
        // a thread's chunks are 16 T bytes apart: its window position advances by sq rows and
        // sr columns per chunk, so only the first position takes a division
        const uint32_t sq = 16u * T / uint32_t(w), sr = 16u * T - sq * uint32_t(w);
        WinPos p = win_pos(h + 16u * uint32_t(tid), w);
        for (uint32_t k = tid; k < chunks; k += T) {
            const uint32_t o = h + 16 * k;
            const uint32_t m = window_bits(rows, H, w, has, y0, x0, p, 16);
            *reinterpret_cast<uint4 *>(out + o) =
                make_uint4(spread4(m), spread4(m >> 4), spread4(m >> 8), spread4(m >> 12));
            if (k + T >= chunks) break;
            p.wx += int(sr);
            p.wy += int(sq);
            if (p.wx >= w) {
                p.wx -= w;
                ++p.wy;
            }
            while (p.wy >= w) {
                p.wy -= w;
                ++p.c;
            }
        }
    }
    // the bytes before the first and after the last full chunk (at most 30), one per thread
    const uint32_t tail = h + 16 * chunks;
    const int loose = int(h + (per - tail));
    for (int i = tid; i < loose; i += T) {
        const uint32_t o = uint32_t(i) < h ? uint32_t(i) : tail + (uint32_t(i) - h);
        out[o] = kStream ? uint8_t((wb[o >> 5] >> (o & 31u)) & 1u)
                         : uint8_t(window_bits(rows, H, w, has, y0, x0, win_pos(o, w), 1));
    }
}

}  // namespace

hipError_t launch_observe(const void *state, int B, int C, int H, int W, int row_bytes, int w,
                          uint8_t *dst, hipStream_t s) {
    const size_t base = (size_t(C) * H * sizeof(uint64_t) + 4 + 15) & ~size_t(15);
    const size_t per = size_t(C) * w * w;
    // the window as a bit string: one bit per output byte, two words of padding
    const size_t sw = per / 32 + 2;
    const size_t with_stream = base + ((sw * 4 + 15) & ~size_t(15));
    // lanes per environment: 16 up to 64 chunks of 16 bytes, 32 up to 1024, else 64 (measured
    // on 16 x 16 maps with C = 6: windows of 10, 20 and 31 cells), as long as the workgroup's
    // staged rows (and, where it fits, the bit string) stay within the LDS budget
    int T = per <= 1024 ? 16 : (per <= 16384 ? 32 : 64);
    while (T < 64 && size_t(256 / T) * base > size_t(kLdsBudget)) T *= 2;
    const bool stream = size_t(256 / T) * with_stream <= size_t(kLdsBudget);
    const size_t region = stream ? with_stream : base;
    const int G = 256 / T;
    const dim3 grid((B + G - 1) / G);
    const size_t lds = size_t(G) * region;
    const int ri = int(region), bi = int(base), si = int(sw);
#define AV_OBSERVE(TT, SS)                                                                   \
    hipLaunchKernelGGL((observe_env<TT, SS>), grid, dim3(256), lds, s, state, B, C, H, W,    \
                       row_bytes, w, dst, ri, bi, si)
    if (T == 16) {
        if (stream) AV_OBSERVE(16, true); else AV_OBSERVE(16, false);
    } else if (T == 32) {
        if (stream) AV_OBSERVE(32, true); else AV_OBSERVE(32, false);
    } else {
        if (stream) AV_OBSERVE(64, true); else AV_OBSERVE(64, false);
    }
#undef AV_OBSERVE
    return hipGetLastError();
}

}  // namespace av
