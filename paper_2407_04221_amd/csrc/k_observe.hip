// Observation kernel: the player-centred window of every environment's current map
// (paper Sec. 2.2.2: a local patch of tiles around the player's position; Table 1 uses
// windows of 5, 10, 20 and 31 cells).
//
// One workgroup per environment (one wave per environment, four to a workgroup, when the
// window has at most 64 rows in all).  Its packed rows are staged in LDS; the first player cell
// in row-major order is found with an LDS atomicMin over rows (then the row's lowest set
// bit).  The environment's C x w x w output bytes are built in LDS one window row per thread
// (one map row read, bits shifted to the window's first column), placed at the same offset
// modulo 16 as their global address, and copied out with aligned 16-byte stores (bytes
// only at the two unaligned ends).  Windows too large for LDS are written byte by byte.
// Window cell (wy, wx) shows map cell (py - w/2 + wy, px - w/2 + wx); cells off the map, and
// the whole window of a map without a player, are 0.
#include "av_internal.h"

namespace av {
namespace {

template <typename RowT>
__device__ inline RowT load_row(const void *base, size_t idx, int row_bytes) {
    if (row_bytes == 2) return static_cast<const uint16_t *>(base)[idx];
    if (row_bytes == 4) return static_cast<const uint32_t *>(base)[idx];
    return static_cast<RowT>(static_cast<const uint64_t *>(base)[idx]);
}

__device__ inline int lowbit(uint64_t v) { return __ffsll(static_cast<unsigned long long>(v)) - 1; }

// Stage the packed rows and find the first player cell; returns (py, px), py = H if none.
// tid / T: this thread's index among the T threads that serve the environment.
__device__ inline void stage_rows(const void *state, int B, int C, int H, int row_bytes, int b,
                                  uint64_t *rows, int *first, int &py, int &px, int tid, int T,
                                  bool live) {
    if (tid == 0) *first = H;
    if (live)
        for (int r = tid; r < C * H; r += T) {
            const int c = r / H, y = r - c * H;
            rows[r] = load_row<uint64_t>(state, (size_t(c) * B + b) * H + y, row_bytes);
        }
    __syncthreads();
    if (live)
        for (int y = tid; y < H; y += T)
            if (rows[size_t(kChPlayer) * H + y]) atomicMin(first, y);
    __syncthreads();
    py = *first;
    px = (live && py < H) ? lowbit(rows[size_t(kChPlayer) * H + py]) : 0;
}

// T threads per environment, 256 / T environments per workgroup, `region` LDS bytes each.
template <int T>
__global__ void __launch_bounds__(256) observe_staged(const void *state, int B, int C, int H, int W,
                                                      int row_bytes, int w, uint8_t *dst,
                                                      int region) {
    extern __shared__ __align__(16) unsigned char lds[];
    const int G = 256 / T;
    const int tid = threadIdx.x % T, slot = threadIdx.x / T;
    const int b = blockIdx.x * G + slot;
    const bool live = b < B;
    unsigned char *base = lds + size_t(slot) * region;
    uint64_t *rows = reinterpret_cast<uint64_t *>(base);   // [C][H]
    int *first = reinterpret_cast<int *>(rows + size_t(C) * H);
    unsigned char *win = base + ((size_t(C) * H * 8 + 4 + 15) & ~size_t(15));
    int py, px;
    stage_rows(state, B, C, H, row_bytes, b, rows, first, py, px, tid, T, live);
    const bool has = py < H;
    const int y0 = py - w / 2, x0 = px - w / 2;
    const size_t per = size_t(C) * w * w;
    uint8_t *out = dst + size_t(live ? b : 0) * per;
    const int shift = int(reinterpret_cast<uintptr_t>(out) & 15);
    unsigned char *mine = win + shift;                       // same offset modulo 16 as out
    if (live)
        for (int q = tid; q < C * w; q += T) {               // one window row per thread
            const int c = q / w, wy = q - c * w, y = y0 + wy;
            const uint64_t row = (has && y >= 0 && y < H) ? rows[size_t(c) * H + y] : 0ull;
            unsigned char *o = mine + size_t(q) * w;
            for (int wx = 0; wx < w; ++wx) {
                const int x = x0 + wx;
                o[wx] = uint8_t(unsigned(x) < unsigned(W) ? (row >> x) & 1ull : 0ull);
            }
        }
    __syncthreads();
    if (!live) return;
    const size_t head = shift ? (16 - shift < per ? size_t(16 - shift) : per) : 0;
    for (size_t i = tid; i < head; i += T) out[i] = mine[i];
    const size_t nch = (per - head) / 16;
    for (size_t k = tid; k < nch; k += T)
        *reinterpret_cast<uint4 *>(out + head + 16 * k) =
            *reinterpret_cast<const uint4 *>(mine + head + 16 * k);
    for (size_t i = head + 16 * nch + tid; i < per; i += T) out[i] = mine[i];
}

__global__ void __launch_bounds__(256) observe_bytes(const void *state, int B, int C, int H, int W,
                                                     int row_bytes, int w, uint8_t *dst) {
    extern __shared__ __align__(16) unsigned char lds[];
    uint64_t *rows = reinterpret_cast<uint64_t *>(lds);   // [C][H]
    int *first = reinterpret_cast<int *>(rows + size_t(C) * H);
    const int b = blockIdx.x, tid = threadIdx.x;
    int py, px;
    stage_rows(state, B, C, H, row_bytes, b, rows, first, py, px, tid, int(blockDim.x), true);
    const bool has = py < H;
    const int y0 = py - w / 2, x0 = px - w / 2;
    const int per = C * w * w;
    uint8_t *out = dst + size_t(b) * per;
    for (int o = tid; o < per; o += blockDim.x) {
        const int c = o / (w * w), rem = o - c * w * w, wy = rem / w, wx = rem - wy * w;
        const int y = y0 + wy, x = x0 + wx;
        uint8_t v = 0;
        if (has && y >= 0 && y < H && x >= 0 && x < W) v = uint8_t((rows[size_t(c) * H + y] >> x) & 1);
        out[o] = v;
    }
}

}  // namespace

hipError_t launch_observe(const void *state, int B, int C, int H, int W, int row_bytes, int w,
                          uint8_t *dst, hipStream_t s) {
    const size_t rows = (size_t(C) * H * sizeof(uint64_t) + 4 + 15) & ~size_t(15);
    const size_t staged = (rows + size_t(C) * w * w + 16 + 15) & ~size_t(15);
    if (C * w <= 64 && 4 * staged <= size_t(kLdsBudget))      // small windows: a wave each
        hipLaunchKernelGGL(observe_staged<64>, dim3((B + 3) / 4), dim3(256), 4 * staged, s, state, B,
                           C, H, W, row_bytes, w, dst, int(staged));
    else if (staged <= size_t(kLdsBudget))
        hipLaunchKernelGGL(observe_staged<256>, dim3(B), dim3(256), staged, s, state, B, C, H, W,
                           row_bytes, w, dst, int(staged));
    else
        hipLaunchKernelGGL(observe_bytes, dim3(B), dim3(256), rows, s, state, B, C, H, W, row_bytes,
                           w, dst);
    return hipGetLastError();
}

}  // namespace av
