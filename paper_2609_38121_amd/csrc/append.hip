// wushkv_append: online key transform, window routing and per-token
// percentile-clipped quantisation into packed pages (Alg. 2 steps 3-4 and
// 7-11; quantiser Eq. (7); windows Sec. 4.4).
//
// One workgroup (256 threads, four waves) owns one tile of up to 64
// consecutive positions of one (sequence, kv head): either a chunk of the
// sink window or exactly one logical page of the quantised region.  Owning a
// whole page means the read-modify-write of shared value-code words never
// races inside a launch.
//
//   phase A  new keys k (bf16) x T_K^T on the 16x16x32 bf16 matrix cores,
//            fp32 accumulate, rounded once to bf16 -> LDS.  Keys that are
//            flushed from the recent ring are copied from it instead.
//            Values (new or ring) -> LDS.
//   phase B  two lanes per (token, K|V) group, half the channels each:
//            exact top-k of |x| with a median-of-three insertion network
//            (each lane over its half, then its partner's list merged in),
//            the type-7 quantile, fp16 scale/zero and the codes.  Key codes
//            go straight to their words; value codes go to LDS.
//   phase C  value-code words (each spans 8 tokens) are assembled from LDS;
//            words only partly covered by this call are merged with what the
//            page already holds.
//   phase D  bf16 window writes (sink and ring) and the optional k~ output.
#include "common.h"
#include "merge.h"
#include "quantise.h"

namespace wushkv {

// Four workgroups per compute unit (their LDS fits four times): the
// registers are held to what four waves per SIMD leave.
template <int D, int BITS, bool ROPE>
__global__ void __launch_bounds__(256, 4) append_kernel(AppendArgs a)
{
    using L = Layout<D, BITS>;
    constexpr int kPitch = D + 8;  // bf16 elements per LDS row (16 B pad)
    __shared__ __attribute__((aligned(16))) uint16_t kt[kPage * kPitch];
    __shared__ __attribute__((aligned(16))) uint16_t vt[kPage * kPitch];
    __shared__ int32_t sh_page[1];  // page index
    __shared__ int32_t sh_cnt[3];   // the sequence's counters (read_counters)

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    // XCD-aware order.  The device hands consecutive workgroups to its 8
    // XCDs in turn (workgroup L runs on XCD L % 8), so the 8 workgroups of a
    // turn take 8 consecutive tiles of one (head, sequence), and the next
    // turns take the same 8 tiles for the other heads and sequences: the
    // rotary-table rows of a tile's positions are read into one XCD's L2 and
    // reused there by every head and sequence.  gridDim.x is a multiple of 8.
    const uint32_t wg = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
    const uint32_t hbs = gridDim.y * gridDim.z, turn = wg / 8;
    const int tile = (int)(8 * (turn / hbs) + wg % 8);
    const int h = (int)((turn % hbs) % gridDim.y), b = (int)((turn % hbs) / gridDim.y);

    // ---- per-sequence bookkeeping (identical in every workgroup)
    const SeqCounters cnt = read_counters(a, b, a.max_new, sh_cnt, tid);
    const int32_t s_old = cnt.s_old, q_old = cnt.q_old, nn = cnt.nn;
    const int32_t s_new = s_old + nn;
    const int32_t q_new = next_quant_end(s_new, q_old, a.s_sink, a.s_keep, a.s_flush);
    const int32_t start_old = q_old > a.s_sink ? q_old : a.s_sink;
    const int32_t first = s_old < start_old ? s_old : start_old;
    const int32_t ring = a.win_slots - a.s_sink;

    // ---- which tile
    int k0 = first < a.s_sink ? (first / kPage) - a.sink_tiles : (first - a.s_sink) / kPage;
    const int k = k0 + tile;
    int32_t blk_lo, blk_hi;
    if (k < 0) {
        blk_lo = (k + a.sink_tiles) * kPage;
        blk_hi = min(blk_lo + kPage, a.s_sink);
    } else {
        blk_lo = a.s_sink + k * kPage;
        blk_hi = blk_lo + kPage;
    }
    const bool do_new = (a.mode & kModeNew) != 0, do_flush = (a.mode & kModeFlush) != 0;
    int32_t lo = max(blk_lo, first), hi = min(blk_hi, s_new);
    if (!do_new) {
        // a flush-only launch touches nothing but the ring positions that
        // are due: [start_old, q_new) below s_old (an empty cache has none)
        lo = max(lo, start_old);
        hi = min(hi, min(s_old, q_new));
    }
    if (lo >= hi) {
        commit_finish(a, b, commit_arrive(a, b, s_old, q_old, nn, tid), s_new, q_new, tid);
        return;
    }

    // position p (lo <= p < hi) is: new if p >= s_old; quantised now if
    // start_old <= p < q_new; otherwise a window entry (sink, or ring if new).
    auto is_new = [&](int32_t p) { return p >= s_old; };
    auto quant_now = [&](int32_t p) {
        return p >= start_old && p < q_new && (is_new(p) ? do_new : do_flush);
    };
    auto window_write = [&](int32_t p) {
        return do_new && is_new(p) && (p < a.s_sink || p >= q_new);
    };

    if (tid == 0) {
        int32_t phys = -1;
        if (k >= 0 && k < a.max_pages) {
            phys = a.page_table[(int64_t)b * a.max_pages + k];
            if (phys < 0 || phys >= a.n_pages) phys = -1;
        }
        sh_page[0] = phys;
    }

    const int64_t head_win = ((int64_t)b * a.n_kv + h) * a.win_slots;  // win_k row base (slots)

    // new values of this tile, loaded early so that their latency overlaps
    // the key transform: first of all, or (with the fused normalisation,
    // whose registers are full until it ends) right after the keys are
    // staged (idx = tid + 256 q is row idx / kVec, 16-byte chunk idx % kVec)
    constexpr int kVec = D / 8;                   // uint4 per row
    constexpr int kVPer = kPage * kVec / 256;     // uint4 per thread
    constexpr int kVRows = 256 / kVec;            // rows between a thread's chunks
    uint4 vpre[kVPer];
    auto load_values = [&]() {
        // the thread's chunks lie kVRows token rows apart in v_new: one
        // element offset, then a constant step (negative for rows before
        // the new ones, which are not loaded)
        const int r0v = tid / kVec, cv = tid % kVec;
        const int64_t step = (int64_t)kVRows * a.n_kv * D;
        const int64_t off0 = (((int64_t)b * a.max_new + (blk_lo + r0v - s_old)) * a.n_kv + h) * D + 8 * cv;
#pragma unroll
        for (int q = 0; q < kVPer; ++q) {
            const int32_t p = blk_lo + r0v + kVRows * q;
            if (p >= lo && p < hi && do_new && is_new(p))
                vpre[q] = *reinterpret_cast<const uint4 *>(a.v_new + (off0 + q * step));
        }
    };
    if constexpr (!ROPE) load_values();

    // ---- phase A: transformed keys -> kt, values -> vt
    // the tile's new positions are [new_lo, hi); window writes go to those
    // below s_sink or at or above q_new
    const int32_t new_lo = max(lo, s_old);
    const bool any_new = do_new && new_lo < hi;
    const bool any_window = any_new && (new_lo < a.s_sink || hi > q_new);
    if (any_new) {
        // Wave w produces output channels [w D/4, (w+1) D/4) for all 64 rows.
        constexpr int kNtW = D / 64;  // N-tiles per wave
        const int j = lane >> 4, n = lane & 15;
        constexpr bool fused = ROPE;
        // this wave's rows of T_K, in flight while the keys are staged (the
        // fused variant loads them after the normalisation: its registers
        // are full until then)
        KeyTile<D, kNtW> xf;
        if constexpr (!fused) xf.load(a.tk, h, wave * kNtW, lane);
        // phase A0: each new row once (wave w rows 16 w .. 16 w + 15, one
        // load per lane and chunk for the whole tile) into the value rows,
        // which serve as the key operand's staging until the values arrive:
        // RoPE(Norm(k)) rounded to bf16 when fused, else k as it came
        // A row that is not new loads the first row of k_new (in bounds;
        // it is replaced by zeros), so that every load of the tile is
        // issued at once, with no branch between them.
        const int r0 = 16 * wave + n;
        const int32_t p0 = blk_lo + r0;
        const bool ld0 = (p0 >= lo && p0 < hi && is_new(p0) && do_new);
        const uint16_t *krow0 =
            a.k_new + (ld0 ? (((int64_t)b * a.max_new + (p0 - s_old)) * a.n_kv + h) * D : (int64_t)0);
        u32x4 kin[L::kChunks];
#pragma unroll
        for (int c = 0; c < L::kChunks; ++c) kin[c] = *reinterpret_cast<const u32x4 *>(krow0 + 32 * c + 8 * j);
        if constexpr (!fused) {
#pragma unroll
            for (int c = 0; c < L::kChunks; ++c) {
                const u32x4 zero = {0u, 0u, 0u, 0u};
                *reinterpret_cast<u32x4 *>(vt + r0 * kPitch + 32 * c + 8 * j) = ld0 ? kin[c] : zero;
            }
        } else {
            const int r = r0;
            const bool ld = ld0;
            float rt[D / 64][16];
            load_rope<D>(a, j, ld ? p0 : 0, rt);
            // (a row that is not new holds the first row of k_new here: its
            // result is replaced by zeros below)
            float x[L::kChunks][8];
#pragma unroll
            for (int c = 0; c < L::kChunks; ++c) {
#pragma unroll
                for (int e = 0; e < 8; ++e) x[c][e] = bf16_bits_to_f32((kin[c][e >> 1] >> (16 * (e & 1))) & 0xFFFFu);
            }
            norm_rope_row<D>(x, j, rt, a);
            load_values();
#pragma unroll
            for (int c = 0; c < L::kChunks; ++c) {
                u32x4 pk;
#pragma unroll
                for (int q = 0; q < 4; ++q) pk[q] = ld ? pack_bf16_rne(x[c][2 * q], x[c][2 * q + 1]) : 0u;
                *reinterpret_cast<u32x4 *>(vt + r * kPitch + 32 * c + 8 * j) = pk;
            }
        }
        __syncthreads();
        if constexpr (fused) xf.load(a.tk, h, wave * kNtW, lane);
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            const int r = 16 * mt + n;  // A row handled by this lane
            bf16x8 aop[L::kChunks];
#pragma unroll
            for (int c = 0; c < L::kChunks; ++c)
                aop[c] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(vt + r * kPitch + 32 * c + 8 * j));
            f32x4 acc[kNtW];
            xf.apply(aop, acc);
#pragma unroll
            for (int nt = 0; nt < kNtW; ++nt) {
                const int ch = (wave * kNtW + nt) * 16 + n;
#pragma unroll
                for (int rr = 0; rr < 4; rr += 2) {
                    uint32_t pr = pack_bf16_rne(acc[nt][rr], acc[nt][rr + 1]);
                    const int row = 16 * mt + 4 * j + rr;
                    kt[row * kPitch + ch] = (uint16_t)(pr & 0xFFFFu);
                    kt[(row + 1) * kPitch + ch] = (uint16_t)(pr >> 16);
                }
            }
        }
        // the value rows are about to be overwritten: every wave must have
        // read its key operands from them
        __syncthreads();
    }
    // The arrival (thread 0) comes after the tile's key and value loads
    // have landed: an atomic on the sequence's count, shared by every tile
    // of the sequence, can take long to return, and the vector memory
    // counter would make every later wait for a load wait for it too.  Its
    // result is needed only at the end.
    const int32_t arrived = commit_arrive(a, b, s_old, q_old, nn, tid);
    // ring-sourced keys (flush) and all values, 16 B per thread-step
    {
#pragma unroll
        for (int q = 0; q < kVPer; ++q) {
            const int idx = tid + 256 * q, r = idx / kVec, cv = idx % kVec;
            const int32_t p = blk_lo + r;
            if (p < lo || p >= hi) continue;
            const bool nw = is_new(p);
            if (nw ? !do_new : !quant_now(p)) continue;
            uint4 vv;
            if (nw) {
                vv = vpre[q];
            } else {
                const int32_t slot = ring_slot(p, a.s_sink, ring);
                const uint16_t *vsrc = a.win_v + (head_win * D) + slot;  // channel-major
                uint16_t e[8];
#pragma unroll
                for (int qq = 0; qq < 8; ++qq) e[qq] = vsrc[(int64_t)(8 * cv + qq) * a.win_slots];
                vv.x = e[0] | ((uint32_t)e[1] << 16);
                vv.y = e[2] | ((uint32_t)e[3] << 16);
                vv.z = e[4] | ((uint32_t)e[5] << 16);
                vv.w = e[6] | ((uint32_t)e[7] << 16);
                *reinterpret_cast<uint4 *>(kt + r * kPitch + 8 * cv) =
                    *reinterpret_cast<const uint4 *>(a.win_k + (head_win + slot) * D + 8 * cv);
            }
            *reinterpret_cast<uint4 *>(vt + r * kPitch + 8 * cv) = vv;
        }
    }
    __syncthreads();
    const int32_t page = sh_page[0];
    uint8_t *pg = page >= 0 ? a.pages + ((int64_t)page * a.n_kv + h) * L::kPageBytes : nullptr;

    // ---- phases B and C
    // quant_now holds for every position of [blk_lo, blk_lo + 64) when the
    // range lies in [lo, hi) and [start_old, q_new), its new positions are
    // appended and its old ones flushed by this launch
    const int32_t blk_end = blk_lo + kPage;
    const bool all_quant = lo <= blk_lo && blk_end <= hi && start_old <= blk_lo && blk_end <= q_new &&
                           (blk_end <= s_old || do_new) && (blk_lo >= s_old || do_flush);
    quantise_tile<D, BITS>(a, kt, vt, blk_lo, [&](int32_t p) { return p >= lo && p < hi && quant_now(p); },
                           all_quant, pg, tid);

    // ---- phase D: bf16 windows and the optional k~ output (a tile of
    // the quantised region of a prefill has neither)
    if (any_window || (any_new && a.k_tilde_out != nullptr)) {
        constexpr int kVec = D / 8;
        for (int idx = tid; idx < kPage * kVec; idx += 256) {
            const int r = idx / kVec, cv = idx % kVec;
            const int32_t p = blk_lo + r;
            if (p < lo || p >= hi || !(do_new && is_new(p))) continue;
            const uint4 kv = *reinterpret_cast<const uint4 *>(kt + r * kPitch + 8 * cv);
            if (a.k_tilde_out != nullptr)
                *reinterpret_cast<uint4 *>(
                    a.k_tilde_out + (((int64_t)b * a.max_new + (p - s_old)) * a.n_kv + h) * D + 8 * cv) = kv;
            if (window_write(p)) {
                const int32_t slot = p < a.s_sink ? p : ring_slot(p, a.s_sink, ring);
                *reinterpret_cast<uint4 *>(a.win_k + (head_win + slot) * D + 8 * cv) = kv;
            }
        }
        // values, channel-major: consecutive threads write consecutive slots
        for (int idx = tid; any_window && idx < kPage * D; idx += 256) {
            const int ch = idx / kPage, r = idx % kPage;
            const int32_t p = blk_lo + r;
            if (p < lo || p >= hi || !window_write(p)) continue;
            const int32_t slot = p < a.s_sink ? p : ring_slot(p, a.s_sink, ring);
            a.win_v[(head_win * D) + (int64_t)ch * a.win_slots + slot] = vt[r * kPitch + ch];
        }
    }
    commit_finish(a, b, arrived, s_new, q_new, tid);
}

// Appends of at most kStepMax tokens per sequence (decode steps): one
// workgroup per (kv head, sequence).  The new keys form one 16-row tile of
// the key transform (KeyTile, the prefill's own operand order: wave w takes
// output channels w D/4 .. w D/4 + D/4 - 1; with the fused normalisation
// and RoPE each wave first applies norm_rope_row to the rows, as the
// prefill does), rounded once to bf16 into LDS; then the newly eligible
// positions are quantised page by page from the ring or from those new rows
// (quantise_tile); last, the new tokens that stay bf16 are written to the
// windows.  Reading the flushed ring slots before writing the new ones makes
// the order independent of the ring's length.
constexpr int kStepMax = 16;

template <int D, int BITS>
__global__ void __launch_bounds__(256) append_step_kernel(AppendArgs a)
{
    using L = Layout<D, BITS>;
    constexpr int kPitch = D + 8;
    constexpr int kNtW = D / 64;  // 16-channel output tiles per wave
    __shared__ __attribute__((aligned(16))) uint16_t kn[kStepMax * kPitch];
    __shared__ __attribute__((aligned(16))) uint16_t kt[kPage * kPitch];
    __shared__ __attribute__((aligned(16))) uint16_t vt[kPage * kPitch];
    __shared__ int32_t sh_page[1];  // page index
    __shared__ int32_t sh_cnt[3];   // the sequence's counters (read_counters)

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int h = blockIdx.x, b = blockIdx.y;
    const SeqCounters cnt = read_counters(a, b, a.max_new, sh_cnt, tid);
    const int32_t s_old = cnt.s_old, q_old = cnt.q_old, nn = cnt.nn;
    const int32_t s_new = s_old + nn;
    const int32_t q_new = next_quant_end(s_new, q_old, a.s_sink, a.s_keep, a.s_flush);
    const int32_t arrived = commit_arrive(a, b, s_old, q_old, nn, tid);
    const int32_t start_old = q_old > a.s_sink ? q_old : a.s_sink;
    const int32_t ring = a.win_slots - a.s_sink;
    const int64_t head_win = ((int64_t)b * a.n_kv + h) * a.win_slots;
    auto new_row = [&](auto *base, int32_t p) {
        return base + (((int64_t)b * a.max_new + (p - s_old)) * a.n_kv + h) * D;
    };

    // ---- transformed new keys -> kn (row t: new token t)
    if (nn > 0) {
        const int j = lane >> 4, n = lane & 15;
        KeyTile<D, kNtW> xf;
        xf.load(a.tk, h, wave * kNtW, lane);
        const bool ld = n < nn;
        const uint16_t *krow = new_row(a.k_new, s_old + (ld ? n : 0));
        bf16x8 aop[L::kChunks];
        u32x4 av[L::kChunks];
#pragma unroll
        for (int c = 0; c < L::kChunks; ++c) {
            av[c] = u32x4{0u, 0u, 0u, 0u};
            if (ld) av[c] = *reinterpret_cast<const u32x4 *>(krow + 32 * c + 8 * j);
        }
        if (a.rope != nullptr) {
            // RoPE(Norm(k)) of row n, rounded to bf16: the prefill's phase A0
            float x[L::kChunks][8];
#pragma unroll
            for (int c = 0; c < L::kChunks; ++c)
#pragma unroll
                for (int e = 0; e < 8; ++e) x[c][e] = bf16_bits_to_f32((av[c][e >> 1] >> (16 * (e & 1))) & 0xFFFFu);
            norm_rope_row<D>(x, j, ld ? s_old + n : 0, a);
#pragma unroll
            for (int c = 0; c < L::kChunks; ++c)
#pragma unroll
                for (int q = 0; q < 4; ++q) av[c][q] = ld ? pack_bf16_rne(x[c][2 * q], x[c][2 * q + 1]) : 0u;
        }
#pragma unroll
        for (int c = 0; c < L::kChunks; ++c) aop[c] = __builtin_bit_cast(bf16x8, av[c]);
        f32x4 acc[kNtW];
        xf.apply(aop, acc);
#pragma unroll
        for (int nt = 0; nt < kNtW; ++nt) {
            const int o = (wave * kNtW + nt) * 16 + n;
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                const int t = 4 * j + rr;
                if (t < nn) {
                    const uint16_t kb = (uint16_t)(pack_bf16_rne(acc[nt][rr], 0.0f) & 0xFFFFu);
                    kn[t * kPitch + o] = kb;
                    if (a.k_tilde_out != nullptr) new_row(a.k_tilde_out, s_old + t)[o] = kb;
                }
            }
        }
    }
    __syncthreads();

    // ---- quantise [start_old, q_new), one page at a time
    if (start_old < q_new)
        flush_range<D, BITS, true>(a, b, h, start_old, q_new, s_old, kn, kt, vt, sh_page, tid);

    // ---- new tokens that stay bf16: sink, or the ring at or after q_new
    for (int t = 0; t < nn; ++t) {
        const int32_t p = s_old + t;
        if (!(p < a.s_sink || p >= q_new)) continue;
        const int32_t slot = p < a.s_sink ? p : ring_slot(p, a.s_sink, ring);
        if (tid < D / 8)
            *reinterpret_cast<uint4 *>(a.win_k + (head_win + slot) * D + 8 * tid) =
                *reinterpret_cast<const uint4 *>(kn + t * kPitch + 8 * tid);
        if (tid < D) a.win_v[(head_win * D) + (int64_t)tid * a.win_slots + slot] = new_row(a.v_new, p)[tid];
    }
    commit_finish(a, b, arrived, s_new, q_new, tid);
}

template <int D, int BITS>
static hipError_t launch_append(const char *name, const AppendArgs &a, dim3 grid, hipStream_t s)
{
    if (a.rope != nullptr) launch(name, append_kernel<D, BITS, true>, grid, dim3(256), s, a);
    else launch(name, append_kernel<D, BITS, false>, grid, dim3(256), s, a);
    return hipGetLastError();
}

// S and S_quant of every sequence advanced after an append launch of many
// tiles, which then counts no arrivals (thousands of workgroups of one
// sequence would queue their device-scope atomics at one address, and each
// holds its slot until its own returns).  Launched after it on the stream,
// so that every tile has read the old values.  One thread per sequence; the
// new-token count is clamped as read_counters clamps it.
__global__ void __launch_bounds__(256) append_commit_kernel(AppendArgs a, int32_t batch)
{
    const int b = (int)(blockIdx.x * 256 + threadIdx.x);
    if (b >= batch) return;
    const int32_t s_old = a.seq_len[b], q_old = a.quant_end[b];
    int32_t nn = a.n_new[b];
    nn = nn < 0 ? 0 : (nn > a.max_new ? a.max_new : nn);
    const int32_t s_new = s_old + nn;
    a.seq_len[b] = s_new;
    a.quant_end[b] = next_quant_end(s_new, q_old, a.s_sink, a.s_keep, a.s_flush);
}

template <int D, int BITS>
static hipError_t launch_append_step(const AppendArgs &a, dim3 grid, hipStream_t s)
{
    launch("append_step_kernel", append_step_kernel<D, BITS>, grid, dim3(256), s, a);
    return hipGetLastError();
}

// ------------------------------------------------------------------ step

// Second launch of wushkv_decode_step.  Workgroups x < n_q merge the
// attention splits of query head x of sequence y (as the decode combine
// does); the n_kv after them then finish Alg. 2 for kv head x - n_q of
// sequence y after its attention: the positions that left the recent window
// are quantised from the ring (steps 7-11), and the last of a sequence's
// workgroups advances its counters.
struct FinishArgs {
    const float *part;  // [batch][n_kv][n_splits][G][D + 2]
    float *out;         // [batch][n_kv G][D]
    int32_t G, n_splits;
};

template <int D, int BITS>
__global__ void __launch_bounds__(256) step_finish_kernel(AppendArgs a, FinishArgs f)
{
    constexpr int kPitch = D + 8;
    __shared__ __attribute__((aligned(16))) uint16_t kt[kPage * kPitch];
    __shared__ __attribute__((aligned(16))) uint16_t vt[kPage * kPitch];
    __shared__ float fw[kMaxSplits];
    __shared__ float red[D];
    __shared__ int32_t sh[4];  // page index, the counters (read_counters)
    const int tid = threadIdx.x, b = blockIdx.y;
    const int n_q = a.n_kv * f.G;
    if ((int)blockIdx.x < n_q) {
        const int qh = blockIdx.x, h = qh / f.G, g = qh % f.G;
        const int64_t stride = (int64_t)f.G * (D + 2);
        const float *pp = f.part + ((int64_t)b * a.n_kv + h) * f.n_splits * stride + g * (D + 2);
        merge_splits<D>(pp, stride, f.n_splits, f.out + ((int64_t)b * n_q + qh) * D, tid, fw, red);
        return;
    }
    const int h = (int)blockIdx.x - n_q;
    const SeqCounters cnt = read_counters(a, b, 1, sh + 1, tid);
    const int32_t s_old = cnt.s_old, q_old = cnt.q_old, nn = cnt.nn;
    const int32_t s_new = s_old + nn;
    const int32_t q_new = next_quant_end(s_new, q_old, a.s_sink, a.s_keep, a.s_flush);
    const int32_t arrived = commit_arrive(a, b, s_old, q_old, nn, tid);
    const int32_t start = q_old > a.s_sink ? q_old : a.s_sink;
    if (start < q_new) flush_range<D, BITS, false>(a, b, h, start, q_new, s_new, kt, kt, vt, sh, tid);
    commit_finish(a, b, arrived, s_new, q_new, tid);
}

}  // namespace wushkv

using namespace wushkv;

// Host-side position of the kappa-quantile (fp64, as in the definition of
// the quantile: pos = kappa (d - 1), lo = floor(pos), t = pos - lo).
static void kappa_position(float kappa, int d, int32_t &lo, float &t)
{
    double pos = (double)kappa * (double)(d - 1);
    double fl = std::floor(pos);
    if (fl < 0.0) fl = 0.0;
    if (fl > (double)(d - 1)) fl = (double)(d - 1);
    lo = (int32_t)fl;
    t = (float)(pos - fl);
}

int wushkv_validate_cache(const wushkv_cache *c);  // api.hip

// The cache's part of the kernel arguments (pointers, sizes, quantiser).
static AppendArgs cache_args(const wushkv_cache *c)
{
    AppendArgs a{};
    a.pages = c->pages;
    a.page_table = c->page_table;
    a.win_k = c->win_k;
    a.win_v = c->win_v;
    a.seq_len = c->seq_len;
    a.quant_end = c->quant_end;
    a.commit = c->commit;
    a.n_kv = c->n_kv_heads;
    a.s_sink = c->s_sink;
    a.s_keep = c->s_keep;
    a.s_flush = c->s_flush;
    a.win_slots = c->win_slots;
    a.max_pages = c->max_pages_per_seq;
    a.n_pages = c->n_pages;
    a.codec = c->codec;
    a.levels = (1 << c->bits) - 1;
    if (c->codec == WUSHKV_CODEC_PCLIP) {
        kappa_position(c->kappa_k, c->head_dim, a.lo_k, a.t_k);
        kappa_position(c->kappa_v, c->head_dim, a.lo_v, a.t_v);
    } else {
        a.quest_coef = 2.0 * (double)c->quest_alpha / (double)((1 << c->bits) - 1);
    }
    a.sink_tiles = (c->s_sink + kPage - 1) / kPage;
    return a;
}

// Both entry points: rope == nullptr appends keys as given; otherwise the
// keys are normalised and rotated first (the caller checked the table).
static int append_impl(const wushkv_cache *c, const uint16_t *k_new, const uint16_t *v_new,
                       const int32_t *n_new, int32_t max_new, const uint16_t *t_k,
                       const float *gain, float eps, const float *rope,
                       uint16_t *k_tilde_out, wushkv_stream_t stream)
{
    int st = wushkv_validate_cache(c);
    if (st != WUSHKV_OK) return st;
    if (max_new < 0) return WUSHKV_EINVAL;
    if (max_new == 0) return WUSHKV_OK;
    if (!k_new || !v_new || !n_new || !t_k) return WUSHKV_EINVAL;

    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    AppendArgs a = cache_args(c);
    a.k_new = k_new;
    a.v_new = v_new;
    a.n_new = n_new;
    a.max_new = max_new;
    a.tk = t_k;
    a.k_tilde_out = k_tilde_out;
    a.gain = gain;
    a.eps = eps;
    a.rope = rope;


    // Tiles a sequence can touch: the sink tiles, plus the span from the
    // oldest unflushed position (at most s_keep + s_flush - 1 back) to the
    // new end.
    const int64_t span = (int64_t)max_new + c->s_keep + c->s_flush - 1;
    // (a multiple of 8: see the tile order in append_kernel; the extra tiles
    // lie past the new end and exit at once)
    const int64_t tiles = (a.sink_tiles + (span + kPage - 1) / kPage + 1 + 7) / 8 * 8;
    if (tiles > 0x7FFFFFFF) return WUSHKV_EINVAL;
    dim3 grid((unsigned)tiles, (unsigned)c->n_kv_heads, (unsigned)c->batch);

    // Flushed ring slots may be reused by new tokens of the same call only if
    // the ring is shorter than the span; then flush first, in its own launch.
    // That launch only touches positions already in the ring, which span at
    // most the ring's length from the first unflushed one.
    const int64_t ring = (int64_t)c->win_slots - c->s_sink;
    const bool fused = ring >= span;
    const dim3 flush_grid((unsigned)std::min<int64_t>(tiles, (a.sink_tiles + (ring + kPage - 1) / kPage + 1 + 7) / 8 * 8),
                          grid.y, grid.z);

    // The launch that appends the new tokens advances the counters (its
    // workgroups are the last to read them): its last arriving workgroup
    // does, or, beyond kArrivalsMax workgroups per sequence, a launch of its
    // own right after it.
    constexpr int64_t kArrivalsMax = 64;
    auto go = [&](int mode) -> hipError_t {
        a.mode = mode;
        const char *name = mode == kModeFlush ? "append_flush" : "append_kernel";
        const dim3 g = mode == kModeFlush ? flush_grid : grid;
        const bool commit_launch = (mode & kModeNew) && (int64_t)g.x * g.y > kArrivalsMax;
        a.arrivals = (mode & kModeNew) && !commit_launch ? (int32_t)(g.x * g.y) : 0;
        const int key = c->head_dim * 10 + storage_bits(c->bits);
        hipError_t e = hipErrorInvalidValue;
        switch (key) {
            case 1282: e = launch_append<128, 2>(name, a, g, s); break;
            case 1284: e = launch_append<128, 4>(name, a, g, s); break;
            case 642: e = launch_append<64, 2>(name, a, g, s); break;
            case 644: e = launch_append<64, 4>(name, a, g, s); break;
        }
        if (e == hipSuccess && commit_launch) {
            launch("append_commit", append_commit_kernel, dim3((unsigned)((c->batch + 255) / 256)), dim3(256), s, a,
                   (int32_t)c->batch);
            e = hipGetLastError();
        }
        return e;
    };
    hipError_t e;
    if (max_new <= kStepMax) {
        const dim3 sgrid((unsigned)c->n_kv_heads, (unsigned)c->batch);
        a.arrivals = (int32_t)sgrid.x;
        const int key = c->head_dim * 10 + storage_bits(c->bits);
        switch (key) {
            case 1282: e = launch_append_step<128, 2>(a, sgrid, s); break;
            case 1284: e = launch_append_step<128, 4>(a, sgrid, s); break;
            case 642: e = launch_append_step<64, 2>(a, sgrid, s); break;
            default: e = launch_append_step<64, 4>(a, sgrid, s); break;
        }
    } else if (fused) {
        e = go(kModeFlush | kModeNew);
    } else {
        e = go(kModeFlush);
        if (e == hipSuccess) e = go(kModeNew);
    }
    if (e != hipSuccess) return WUSHKV_ELAUNCH;
    return WUSHKV_OK;
}

extern "C" int wushkv_append(const wushkv_cache *c, const uint16_t *k_new, const uint16_t *v_new,
                             const int32_t *n_new, int32_t max_new, const uint16_t *t_k,
                             uint16_t *k_tilde_out, wushkv_stream_t stream)
{
    return append_impl(c, k_new, v_new, n_new, max_new, t_k, nullptr, 0.0f, nullptr, k_tilde_out,
                       stream);
}

extern "C" int wushkv_append_norm_rope(const wushkv_cache *c, const uint16_t *k_raw,
                                       const uint16_t *v_new, const int32_t *n_new,
                                       int32_t max_new, const uint16_t *t_k,
                                       const float *norm_gain, float norm_eps,
                                       const float *rope_table, int32_t rope_positions,
                                       uint16_t *k_tilde_out, wushkv_stream_t stream)
{
    int st = wushkv_validate_cache(c);
    if (st != WUSHKV_OK) return st;
    if (rope_table == nullptr || !(norm_eps >= 0.0f) || norm_eps == INFINITY) return WUSHKV_EINVAL;
    if ((int64_t)rope_positions < (int64_t)c->max_pages_per_seq * kPage + c->s_sink) return WUSHKV_EINVAL;
    if (((uintptr_t)rope_table | (uintptr_t)norm_gain) & 15u) return WUSHKV_EINVAL;
    return append_impl(c, k_raw, v_new, n_new, max_new, t_k, norm_gain, norm_eps, rope_table,
                       k_tilde_out, stream);
}

// The finishing launch of wushkv_decode_step (its attention launch precedes
// it on the stream): see step_finish_kernel.  Declared in decode.hip.
int wushkv_step_finish(const wushkv_cache *c, const int32_t *n_new, const float *part, float *out,
                       int32_t G, int32_t n_splits, hipStream_t s)
{
    AppendArgs a = cache_args(c);
    a.n_new = n_new;
    a.max_new = 1;
    a.arrivals = c->n_kv_heads;  // the flush workgroups of a sequence
    FinishArgs f{part, out, G, n_splits};
    const dim3 grid((unsigned)(c->n_kv_heads * G + c->n_kv_heads), (unsigned)c->batch);
    const int key = c->head_dim * 10 + storage_bits(c->bits);
    switch (key) {
        case 1282: launch("step_finish_kernel", step_finish_kernel<128, 2>, grid, dim3(256), s, a, f); break;
        case 1284: launch("step_finish_kernel", step_finish_kernel<128, 4>, grid, dim3(256), s, a, f); break;
        case 642: launch("step_finish_kernel", step_finish_kernel<64, 2>, grid, dim3(256), s, a, f); break;
        default: launch("step_finish_kernel", step_finish_kernel<64, 4>, grid, dim3(256), s, a, f); break;
    }
    return hipGetLastError() == hipSuccess ? WUSHKV_OK : WUSHKV_ELAUNCH;
}
