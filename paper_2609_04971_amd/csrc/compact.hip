// (a5) In-place, order-preserving compaction of K and V for gfx950:
// row i <- row kept[i] for i < n (Section 2.2, Eq. 8; Algorithm 2, Gather
// after Sort).  HBM-bound: every moved row is read once and written once.
//
// kept is strictly ascending, so kept[i] >= i: a row only ever moves
// towards the front.  Work items are segments of kSegRows destination rows;
// each head's workgroups take their segment numbers from a per-head ticket,
// so segments of a head start in order.  A segment first loads all of its
// source rows into registers and publishes "read done"; before writing it
// waits for every lower segment of the same head whose source range meets
// its destination rows (row x is read only by the segment holding the kept
// index x, and kept[j] >= j puts that segment at or below this one).  With
// a sparse selection that is about one segment, started long before.  Those segments hold lower tickets, have started, and
// publish before they wait, so the waits always end.  Rows already in
// place (kept[i] == i) are neither read nor written.
//
// The hazard is write-after-read only (no segment reads a row another
// segment writes), so the hand-off needs no cache maintenance: a segment's
// loads have returned before its flag is stored, and a writer stores only
// after it has seen the flag.
#include "device_common.h"
#include "internal.h"

namespace bkv {
namespace {

constexpr int kThreads = 256;

struct Args {
    char* K;
    char* V;
    const int32_t* kept;
    int* hdr;
    int* hctl;   // [P][kHcWords] per-head control lines
    int* flags;  // [P][nseg] read-done flags
    int P, budget, N, n_keep, nseg, total;
    size_t head_stride;  // bytes between heads (N_cap * row bytes)
};

// RB = row bytes (D * element size); VPR = 16-byte vectors per row.
template <int RB>
__global__ __launch_bounds__(kThreads) void compact_kernel(Args a) {
    constexpr int VPR = RB / 16;
    constexpr int NV = 2 * kSegRows * VPR / kThreads;  // vectors per thread (K and V)
    __shared__ int s_ticket, s_ok, s_move, s_bad, s_wait_ok, s_last;
    __shared__ int s_src[kSegRows];
    const int tid = threadIdx.x;
    const int h = blockIdx.x / a.nseg;
    int* hc = a.hctl + (size_t)h * kHcWords;
    if (tid == 0) {
        // ticket and stamp requested together (the stamp as one 16-byte
        // load); a ticket taken on a bad workspace is never used
        const int t = dev::fetch_add_relaxed(hc + kHcCpTicket, 1);
        const dev::u32x4 hdr = *reinterpret_cast<const dev::u32x4*>(a.hdr);
        s_ok = hdr[kHdrMagic] == kWsMagic && (int)hdr[kHdrP] == a.P && (int)hdr[kHdrBudget] == a.budget;
        s_ticket = t;
        if (!s_ok) dev::raise_error(a.hdr, kErrStamp);
        s_move = 0;
        s_bad = 0;
        s_wait_ok = 1;
    }
    __syncthreads();
    if (!s_ok) return;
    if (s_ticket >= a.nseg) {  // control block was not clear: do nothing
        if (tid == 0) dev::raise_error(a.hdr, kErrStamp);
        return;
    }
    const int seg = s_ticket;  // segments of a head start in ticket order
    const int i0 = seg * kSegRows;
    const int rows = min(kSegRows, a.n_keep - i0);
    const int32_t* kh = a.kept + (size_t)h * a.n_keep;
    if (tid < rows) {
        const int src = kh[i0 + tid];
        s_src[tid] = src;
        if (src != i0 + tid) s_move = 1;  // benign race: any writer stores 1
        // not a strictly ascending index into [0, N): the hazard waits below
        // rely on every segment's sources lying in [first, last] of its own
        if (src < i0 + tid || src >= a.N || (i0 + tid > 0 && src <= kh[i0 + tid - 1])) s_bad = 1;
    }
    __syncthreads();
    if (s_bad && tid == 0) dev::raise_error(a.hdr, kErrBadIndex);
    const bool move = s_move != 0 && !s_bad;
    char* Kh = a.K + (size_t)h * a.head_stride;
    char* Vh = a.V + (size_t)h * a.head_stride;

    // Rows are read once and written once: both go non-temporal, which
    // measured about 9 % faster on the 32K layer than the default policy.
    dev::u32x4 buf[NV];
    if (move) {
        dev::static_for<NV>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            const int e = tid + k * kThreads;        // vector index within the segment
            const int which = e / (kSegRows * VPR);  // 0 = K, 1 = V
            const int r = (e / VPR) % kSegRows, v = e % VPR;
            if (r < rows && s_src[r] != i0 + r) {
                const char* base = which ? Vh : Kh;
                buf[k] = __builtin_nontemporal_load(reinterpret_cast<const dev::u32x4*>(base + (size_t)s_src[r] * RB) + v);
            }
        });
    }
    // Every load of the workgroup has returned before the flag goes up.
    dev::wait_all_memory();
    __syncthreads();
    if (tid == 0) dev::st_flag(a.flags + (size_t)h * a.nseg + seg, 1);
    if (move) {
        // Wait for the lower segments whose source rows [first, last] meet
        // our destination rows [i0, i0 + rows): row x is read only by the
        // segment holding the kept index x, which is at or below ours.
        if (tid < 64) {
            for (int sp = tid; sp < seg; sp += 64) {
                const int first_src = kh[sp * kSegRows];
                const int last_src = kh[min((sp + 1) * kSegRows, a.n_keep) - 1];
                const bool meets = last_src >= i0 && first_src < i0 + rows;
                if (meets) {
                    if (!dev::wait_flag(a.flags + (size_t)h * a.nseg + sp)) {
                        s_wait_ok = 0;
                        dev::raise_error(a.hdr, kErrCompactWait);
                    }
                }
            }
        }
        __syncthreads();
        if (s_wait_ok) {
            dev::static_for<NV>([&](auto kc) {
                constexpr int k = decltype(kc)::value;
                const int e = tid + k * kThreads;
                const int which = e / (kSegRows * VPR);
                const int r = (e / VPR) % kSegRows, v = e % VPR;
                if (r < rows && s_src[r] != i0 + r) {
                    char* base = which ? Vh : Kh;
                    __builtin_nontemporal_store(buf[k], reinterpret_cast<dev::u32x4*>(base + (size_t)(i0 + r) * RB) + v);
                }
            });
        }
    }
    // The last item to finish clears the control block for the next launch.
    __syncthreads();
    if (tid == 0) s_last = (dev::fetch_add_relaxed(hc + kHcCpDone, 1) == a.nseg - 1);
    __syncthreads();
    if (s_last) {  // every segment of the head is done: clear its control words
        for (int i = tid; i < a.nseg; i += kThreads) dev::st_flag(a.flags + (size_t)h * a.nseg + i, 0);
        if (tid == 0) {
            dev::st_flag(hc + kHcCpTicket, 0);
            dev::st_flag(hc + kHcCpDone, 0);
        }
    }
}

}  // namespace

hipError_t launch_compact(const bkv_dims& d, const WsLayout& L, void* K, void* V, const int32_t* kept, void* ws,
                          hipStream_t s) {
    char* w = static_cast<char*>(ws);
    Args a;
    a.K = static_cast<char*>(K);
    a.V = static_cast<char*>(V);
    a.kept = kept;
    a.hdr = reinterpret_cast<int*>(w);
    a.hctl = reinterpret_cast<int*>(w + L.hctl);
    a.flags = reinterpret_cast<int*>(w + L.cflags);
    a.P = L.P;
    a.budget = d.budget;
    a.N = d.N;
    a.n_keep = d.N < d.budget ? d.N : d.budget;
    a.nseg = (a.n_keep + kSegRows - 1) / kSegRows;
    a.total = a.P * a.nseg;
    const int es = d.dtype == BKV_BF16 ? 2 : 4;
    const int rb = d.D * es;
    a.head_stride = (size_t)d.N_cap * rb;
    if (a.total == 0) return hipSuccess;
    switch (rb) {
        case 128: hipLaunchKernelGGL(compact_kernel<128>, dim3(a.total), dim3(kThreads), 0, s, a); break;
        case 256: hipLaunchKernelGGL(compact_kernel<256>, dim3(a.total), dim3(kThreads), 0, s, a); break;
        default: hipLaunchKernelGGL(compact_kernel<512>, dim3(a.total), dim3(kThreads), 0, s, a); break;
    }
    return hipGetLastError();
}

}  // namespace bkv
