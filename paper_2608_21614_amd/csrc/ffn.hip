// ffn.hip -- grouped SwiGLU expert FFN over the resident and shared experts
// (SAEM Section IV-D.2: resident experts on the matrix cores; Section IV-E.1:
// one batched execution per expert over its contiguous, repacked rows).
//
// Row space of the expert outputs: packed rows [0, T*k) (resident experts
// first, see repack.hip), then the rows of shared expert s at T*k + s*T + t.
//   phase 1: act[p, f] = silu(x[tok(p)] . W1[:,f]) * (x[tok(p)] . W3[:,f])
//   phase 2: y[c][p, h] = sum over K chunk c of act[p, :] . W2[:,h]
//
// Expert weights are in the MFMA tile layout (pack.hip): a 16-row x 32-column
// block is 1 KB of contiguous memory whose 64 16-byte pieces are the 64 lanes'
// MFMA A operands.
//
// Two kernel families:
//  * stream  (T <= 64, decode, and fp32 prefill; bf16 MFMA 16x16x32, fp32 MFMA
//    16x16x4): at decode the weights are streamed from HBM exactly once.  A
//    workgroup owns 32 features (phase 1: 32 gate + 32 up weight rows) or 64
//    outputs (phase 2: 64 rows of W2) of one expert; the weights are the MFMA
//    M side and the expert's tokens the N side, in tiles of 16.  Its four waves
//    split K interleaved -- wave w takes the 32-wide K steps w, w+4, w+8, ... --
//    so at any moment the workgroup reads 4 KB of contiguous memory per weight
//    tile; each wave double-buffers its loads in registers (the next two K
//    steps are in flight while the MFMAs of the current two run).  In the bf16
//    kernels a group whose rows fill one or two 16-row tiles runs a copy of the
//    K loop built for that many, whatever the kernel's tile count.  The waves'
//    partial tiles are summed through LDS in wave order.  Phase 2 also splits K
//    across workgroups into `ks` chunks whose partial sums the combine adds in
//    fixed order.  SwiGLU is applied in the phase-1 epilogue, so the gate and up
//    projections are never stored.  fp32 batches with T > 64 run this kernel on
//    chunks of 64 rows of a group: an item is then (group, weight rows, chunk),
//    found from a prefix over the active groups that every workgroup computes.
//    In the fused forward at decode, phase 1 also does the repacking: its
//    workgroups count the top-k ids themselves (the batch is at most 512 pairs)
//    and look their group's tokens up in them, one extra workgroup writes the
//    repack's outputs for phase 2 and the combine, and phase 2's trailing
//    workgroups pack the offloaded rows.  That saves the repack's launch and
//    its chain of dependent memory round trips before the weights start to flow.
//  * tiled   (bf16, T > 64, prefill): 256 x 256 output tiles (eight waves of
//    128 x 64 on MFMA 32x32x16) that one workgroup per CU works through in
//    turn, both operands read as 1 KB tile-layout blocks by direct global->LDS
//    loads through a five-stage ring; a token gather first copies the resident
//    groups' rows into that layout, and phase 1 writes the activations in it;
//    the expert outputs are bf16.
// Both read counts and offsets from device memory: the stream kernel's grid is
// sized for the worst case on the host and surplus workgroups exit at once; the
// tiled kernel runs one workgroup per CU.
#include <type_traits>

#include "block_ops.hpp"
#include "common.hpp"
#include "kernels.hpp"

namespace saem {
namespace {

struct Args {
    int T, H, E, F, k, S, Fs, slots;
    const void* x;
    const int32_t* perm;
    const int32_t* counts;
    const int32_t* seg_start;
    const int32_t* expert_slot;
    const void* w13;
    const void* w2;
    const void* ws13;
    const void* ws2;
    void* act;
    int Fa;
    float* y;
    int ks;
    long long y_ks_stride;
    int max_routed;   // routed groups the grid reserves (>= active resident experts)
    int ipg_r;        // items (workgroups) per routed group
    int ipg_s;        // items per shared group
    int chunked;      // stream kernel: items cover the groups' rows in chunks of 64 (fp32 prefill)
    // offloaded-row pack done by the workgroups past the FFN items (phase 1; phase 2
    // in the fused path)
    const float* topk_w;
    const int32_t* n_res;
    void* off_rows;
    float* off_w;
    void* xg;         // bf16 prefill: gathered token rows in the tile layout
    int32_t* tmeta;   // bf16 prefill: item tables of the tiled kernels
    int tcap1;        // capacity of the phase-1 table
    uint16_t* y16;    // bf16 prefill: expert outputs [rows][H] in bf16 (instead of y)
    // decode with the repacking in phase 1 (fused): the ids, and the repack's outputs
    int fused;
    int slot_items;   // fused phase 1: routed item gi is slot gi's expert (every slot can be active)
    const int32_t* topk_idx;
    int32_t* rp_counts;
    int32_t* rp_seg_start;
    int32_t* rp_perm;
    int32_t* rp_inv_perm;
    int32_t* rp_n_res;
};

// off_rows[p - n_res] = x[perm[p] / k] and off_w[p - n_res] = topk_w[perm[p]] for the
// offloaded rows p = n_res + wg, n_res + wg + nwg, ...
__device__ void pack_offloaded(const Args& a, int wg, int nwg, int elt) {
    const int P = a.T * a.k;
    const int nres = *a.n_res;
    const int chunks = a.H * elt / 16;  // 16-byte chunks of a row
    for (int p = nres + wg; p < P; p += nwg) {
        const int q = a.perm[p];
        if (q < 0 || q >= P) continue;
        const int t = q / a.k;
        if (a.off_rows) {
            const u32x4* src = reinterpret_cast<const u32x4*>(static_cast<const uint8_t*>(a.x) + (size_t)t * a.H * elt);
            u32x4* dst = reinterpret_cast<u32x4*>(static_cast<uint8_t*>(a.off_rows) + (size_t)(p - nres) * a.H * elt);
            for (int c = threadIdx.x; c < chunks; c += blockDim.x) dst[c] = src[c];
        }
        if (a.off_w && threadIdx.x == 0) a.off_w[p - nres] = a.topk_w[q];
    }
}

// One group of rows: a resident routed expert or a shared expert.
struct Group {
    int rowbase;   // first row in the row space
    int count;     // rows
    int routed;    // 1: rows are packed pairs (token = perm[p] / k); 0: row n is token n
    int Fg;        // expert width
    const uint8_t* w13;
    const uint8_t* w2;
};

// Active resident routed experts (ascending id) into s_list; returns their number.
// With s_info, entry i also gets expert s_list[i]'s (segment start, count, slot),
// read in the same round trip as the counts.
// Must be called by all threads of a 256-thread workgroup.
__device__ int list_active(const Args& a, int* s_list, int* s_wsum, int4* s_info = nullptr) {
    const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
    const int e = tid;
    bool act = false;
    int sl = -1, cnt = 0, seg = 0;
    if (e < a.E) {
        sl = a.expert_slot[e];
        cnt = a.counts[e];
        if (s_info) seg = a.seg_start[e];
        act = is_resident(sl, a.slots) && cnt > 0;
    }
    const unsigned long long b = __ballot(act);
    if (lane == 0) s_wsum[wave] = __popcll(b);
    __syncthreads();
    int base = 0;
    for (int w = 0; w < wave; ++w) base += s_wsum[w];
    if (act) {
        const int pos = base + __popcll(b & ((1ull << lane) - 1ull));
        s_list[pos] = e;
        if (s_info) s_info[pos] = make_int4(seg, cnt, sl, 0);
    }
    const int n = s_wsum[0] + s_wsum[1] + s_wsum[2] + s_wsum[3];
    __syncthreads();
    return n;
}

// list_active for a phase-1 workgroup of the fused decode path, where no repack has
// run yet: the counts come from the top-k ids (P = T k <= 512 pairs, two per thread,
// ids outside [0, E) dropped), and one wave scans them in group order -- resident
// experts by id, then offloaded ones -- into segment starts, as the repack does, and
// compacts the active resident experts in the same pass.  The list, counts and starts
// are the ones list_active reads after a repack.  *id0 / *id1: this thread's ids (pairs
// tid and tid + 256, -1 past P), for group_rows_from_ids.  s_scr: 513 ints of LDS.
// The three loads it needs are PrologueIds, which a caller may issue early.
struct PrologueIds {
    int q0, q1, slot;  // raw top-k ids of pairs tid, tid + 256; expert_slot[tid]
};
__device__ __forceinline__ PrologueIds load_prologue_ids(const Args& a) {
    const int tid = threadIdx.x, P = a.T * a.k;
    PrologueIds p;
    // no branch around the loads, so that a caller's later loads can stay in flight while
    // these are waited for
    const int sl = a.expert_slot[tid < a.E ? tid : 0];
    p.slot = tid < a.E ? sl : -1;
    p.q0 = a.topk_idx[tid < P ? tid : 0];
    p.q1 = a.topk_idx[tid + 256 < P ? tid + 256 : 0];
    return p;
}
__device__ int list_active_from_ids(const Args& a, const PrologueIds& ld, int* s_list, int4* s_info, int* s_scr,
                                    int* id0, int* id1) {
    int* s_cnt = s_scr;         // [256] pairs per expert
    int* s_slot = s_scr + 256;  // [256] slot of each expert (-1 past E)
    int* s_n = s_scr + 512;     // [1] active experts
    const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
    const int P = a.T * a.k;
    s_cnt[tid] = 0;
    s_slot[tid] = ld.slot;
    const int q0 = ld.q0, q1 = ld.q1;
    *id0 = (tid < P && q0 >= 0 && q0 < a.E) ? q0 : -1;
    *id1 = (tid + 256 < P && q1 >= 0 && q1 < a.E) ? q1 : -1;
    __syncthreads();
    if (*id0 >= 0) atomicAdd(&s_cnt[*id0], 1);
    if (*id1 >= 0) atomicAdd(&s_cnt[*id1], 1);
    __syncthreads();
    if (wave == 0) {
        int cnt[4], sl[4];
        bool res[4];
        int rs = 0, os = 0, ac = 0;  // lane owns experts 4 lane .. 4 lane + 3
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = 4 * lane + i;
            cnt[i] = s_cnt[e];
            sl[i] = s_slot[e];
            res[i] = e < a.E && is_resident(sl[i], a.slots);
            if (res[i]) rs += cnt[i];
            else os += cnt[i];
            if (res[i] && cnt[i] > 0) ++ac;
        }
        int rinc = rs, oinc = os, ainc = ac;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int x = __shfl_up(rinc, off, 64), y = __shfl_up(oinc, off, 64), z = __shfl_up(ainc, off, 64);
            if (lane >= off) {
                rinc += x;
                oinc += y;
                ainc += z;
            }
        }
        const int rtot = __shfl(rinc, 63, 64);
        int rp = rinc - rs, op = rtot + (oinc - os), pos = ainc - ac;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = 4 * lane + i;
            const int start = res[i] ? rp : op;
            if (res[i]) rp += cnt[i];
            else op += cnt[i];
            if (res[i] && cnt[i] > 0) {
                s_list[pos] = e;
                s_info[pos] = make_int4(start, cnt[i], sl[i], 0);
                ++pos;
            }
        }
        if (lane == 63) *s_n = ainc;
    }
    __syncthreads();
    return *s_n;
}

// The tokens of expert e's pairs in index order (its rows in the packed order), from the
// ids list_active_from_ids left in registers: s_tok[n] = token of row n.  s_w8: 8 ints.
__device__ void group_rows_from_ids(int e, int k, int id0, int id1, int* s_tok, int* s_w8) {
    const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
    const unsigned long long m0 = __ballot(id0 == e), m1 = __ballot(id1 == e);
    if (lane == 0) {
        s_w8[wave] = __popcll(m0);
        s_w8[4 + wave] = __popcll(m1);
    }
    __syncthreads();
    int b0 = 0, b1 = 0;
    for (int w = 0; w < 4; ++w) {
        b1 += s_w8[w];
        if (w < wave) {
            b0 += s_w8[w];
            b1 += s_w8[4 + w];
        }
    }
    const unsigned long long lt = (1ull << lane) - 1ull;
    // an expert appears at most once per token, so a group holds at most T <= 64 rows
    const int r0 = b0 + __popcll(m0 & lt), r1 = b1 + __popcll(m1 & lt);
    if (id0 == e && r0 < 64) s_tok[r0] = tid / k;
    if (id1 == e && r1 < 64) s_tok[r1] = (tid + 256) / k;
    __syncthreads();
}

// Routed group from its expert's segment start, count and slot.
__device__ Group routed_group_of(const Args& a, int rb, int c, int slot_, size_t elt) {
    Group g;
    const int P = a.T * a.k;
    rb = rb < 0 ? 0 : (rb > P ? P : rb);
    c = c < 0 ? 0 : (c > P - rb ? P - rb : c);
    g.rowbase = rb;
    g.count = c;
    g.routed = 1;
    g.Fg = a.F;
    const size_t slot = (size_t)slot_;
    g.w13 = static_cast<const uint8_t*>(a.w13) + slot * 2 * a.F * a.H * elt;
    g.w2 = static_cast<const uint8_t*>(a.w2) + slot * a.H * a.F * elt;
    return g;
}

__device__ Group routed_group(const Args& a, int e, size_t elt) {
    return routed_group_of(a, a.seg_start[e], a.counts[e], a.expert_slot[e], elt);
}

__device__ Group shared_group(const Args& a, int s, size_t elt) {
    Group g;
    g.rowbase = a.T * a.k + s * a.T;
    g.count = a.T;
    g.routed = 0;
    g.Fg = a.Fs;
    g.w13 = static_cast<const uint8_t*>(a.ws13) + (size_t)s * 2 * a.Fs * a.H * elt;
    g.w2 = static_cast<const uint8_t*>(a.ws2) + (size_t)s * a.H * a.Fs * elt;
    return g;
}

// Token of row n of a group, or -1 when out of range.
__device__ __forceinline__ int group_token(const Args& a, const Group& g, int n) {
    if (n >= g.count) return -1;
    int t;
    if (g.routed) {
        const int q = a.perm[g.rowbase + n];
        t = (q >= 0) ? q / a.k : -1;
    } else {
        t = n;
    }
    return (t >= 0 && t < a.T) ? t : -1;
}

constexpr int kGMaxGroups = 264;  // 256 routed + 8 shared

// s_out[g] = sum_{g' < g} f(g') for g < n (n <= kGMaxGroups), s_out[n] = the total,
// which is also returned; wave 0 scans, every thread of the workgroup must call.
// *s_tot must not be read by any thread between its previous use and this call.
template <typename Fn>
__device__ int group_prefix(int n, int* s_out, int* s_tot, Fn f) {
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        constexpr int PER = (kGMaxGroups + 63) / 64;
        int v[PER], sum = 0;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int gi = PER * lane + i;
            v[i] = gi < n ? f(gi) : 0;
            sum += v[i];
        }
        int inc = sum;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int o = __shfl_up(inc, off, 64);
            if (lane >= off) inc += o;
        }
        int run = inc - sum;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int gi = PER * lane + i;
            if (gi < n) s_out[gi] = run;
            run += v[i];
        }
        if (lane == 63) {
            s_out[n] = inc;
            *s_tot = inc;
        }
    }
    __syncthreads();
    return *s_tot;
}

// ---------------------------------------------------------------------------
// stream kernel (decode, fp32 prefill)
// ---------------------------------------------------------------------------

// 16-row weight tiles per stream workgroup: two with a single token tile (twice
// the workgroups, for the small grids of the smallest batches), else four.
constexpr int stream_mt(int nt) { return nt == 1 ? 2 : 4; }

// kStreamW: the weights are loaded non-temporally (they do not stay in the
// caches for a later use), which raises the streaming rate when the call's
// weights are far larger than the caches; small weight sets that stay in the
// MALL between calls are read with plain loads.
// The bound of two workgroups per CU keeps every instance at two waves per SIMD: fp32
// operands double the fragment registers, and the one-tile copy of the K loop (below)
// adds registers to the wider bf16 instances; without the bound both would drop to one.
template <typename Elt, int NT, bool kDown, bool kStreamW>
__global__ void __launch_bounds__(256, 2) k_ffn_stream(Args a) {
    using F8 = Frag8<Elt>;
    constexpr int MT = stream_mt(NT);              // 16-row weight tiles per workgroup
    constexpr int MH = MT / 2;                     // phase 1: gate tiles (then as many up tiles)
    constexpr int U = sizeof(Elt) == 2 ? 2 : 1;    // K steps per load batch (two batches in flight)
    __shared__ int s_list[256];
    __shared__ int s_wsum[8];
    __shared__ int4 s_info[256];
    // the epilogue's partial tiles, or the repack's LDS in the fused path's repack
    // workgroup (which never reaches the epilogue).  The fused prologue's scratch has
    // its own arrays: a wave with no K steps of its own writes its partial tiles while
    // the other waves may still read the group's token rows.
    constexpr int kRedBytes = 4 * MT * NT * kWave * 16;
    constexpr int kRepackBytes = repack_lds_ints<256>() * 4;
    __shared__ __attribute__((aligned(16))) uint8_t s_raw[kRedBytes > kRepackBytes ? kRedBytes : kRepackBytes];
    auto& s_red = *reinterpret_cast<f32x4 (*)[4][MT][NT][kWave]>(s_raw);
    __shared__ int s_scr[513];  // fused prologue: pairs and slot per expert, active experts
    __shared__ int s_gtok[64];  // fused prologue: the group's token rows
    __shared__ int s_ipre[kGMaxGroups + 1];
    __shared__ int s_tot;
    __shared__ int s_pos;  // slot-mapped items: the slot's place in the active list

    const int item = blockIdx.x;
    const int n_items = a.max_routed * a.ipg_r + a.S * a.ipg_s;
    if (!a.chunked && item >= n_items) {
        if (a.fused && !kDown) {  // the fused path's repack: one workgroup, P <= 512
            if (item == n_items)
                repack_chunks<256>(a.T, a.E, a.k, a.slots, 0, (a.T * a.k + 255) / 256, a.topk_idx, a.expert_slot,
                                   a.rp_counts, a.rp_seg_start, a.rp_perm, a.rp_inv_perm, a.rp_n_res,
                                   reinterpret_cast<int*>(s_raw));
        } else if (a.fused == (int)kDown) {  // trailing workgroups pack the offloaded rows
            pack_offloaded(a, item - n_items, gridDim.x - n_items, sizeof(Elt));
        }
        return;
    }
    const int wave = threadIdx.x >> 6, lane = lane_id();
    const int r = lane & 15, kq = (lane >> 4) * 8;

    // A shared expert's item needs no active list (its group is known), so it starts
    // streaming its weights without the prologue's dependent round trips.  So does a routed
    // item of the fused phase 1 when every slot can hold an active expert: item gi then
    // takes slot gi, whose weights are known at once, and issues its first weight batch
    // before the prologue finds the slot's expert, its rows and its tokens.
    const bool shared_item = !a.chunked && item < a.S * a.ipg_s;
    const bool by_slot = !a.chunked && a.fused && !kDown && a.slot_items && !shared_item;
    Group g;
    int sub = 0, n0 = 0;  // n0: first row of the group this item covers
    int slot = -1;
    if (shared_item) {
        g = shared_group(a, item / a.ipg_s, sizeof(Elt));
        sub = item % a.ipg_s;
    } else if (by_slot) {
        const int i2 = item - a.S * a.ipg_s;
        slot = i2 / a.ipg_r;
        g = routed_group_of(a, 0, 0, slot, sizeof(Elt));  // rows set after the prologue
        sub = i2 % a.ipg_r;
        if (threadIdx.x == 0) s_pos = INT_MAX;  // read after the prologue's barriers
    }

    // weight tiles of this workgroup (16-row tiles in the tile layout) and the K chunk
    const Elt* wp[MT];
    int row0 = 0, kc = 0, c0 = 0, c1 = 0, n_my = 0, sbase = 0, nb = 0;
    auto setup_weights = [&]() {
        if (!kDown) {
            const int f0 = sub * 16 * MH;
            row0 = f0;
            const int nst = a.H / 32;
            const Elt* w = reinterpret_cast<const Elt*>(g.w13);
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                const int rt = (m < MH ? 0 : g.Fg / 16) + f0 / 16 + m % MH;  // gate tiles, then up tiles
                wp[m] = w + (size_t)rt * nst * 512 + lane * 8;
            }
            c0 = 0;
            c1 = nst;
        } else {
            const int h0 = (sub / a.ks) * 16 * MT;
            kc = sub % a.ks;
            row0 = h0;
            const int nst = g.Fg / 32;
            const Elt* w = reinterpret_cast<const Elt*>(g.w2);
#pragma unroll
            for (int m = 0; m < MT; ++m) wp[m] = w + (size_t)(h0 / 16 + m) * nst * 512 + lane * 8;
            c0 = kc * nst / a.ks;
            c1 = (kc + 1) * nst / a.ks;
        }
        // this wave's K steps: c0 + wave + 4 i
        n_my = (c1 - c0 > wave) ? (c1 - c0 - wave + 3) / 4 : 0;
        sbase = c0 + wave;
        nb = n_my / U;
    };
    // batch b holds this wave's steps i = U*b .. U*b+U-1
    auto load_w = [&](F8 (&A)[U][MT], int b) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int s = sbase + 4 * (U * b + u);
#pragma unroll
            for (int m = 0; m < MT; ++m)
                A[u][m] = kStreamW ? load_frag_stream(wp[m] + (size_t)s * 512) : load_frag(wp[m] + (size_t)s * 512);
        }
    };
    F8 A0[U][MT], A1[U][MT];
    const bool early = shared_item || by_slot;  // weights known before the prologue
    int id0 = -1, id1 = -1, nact = 0;
    if (by_slot) {
        // the prologue's loads first, then the weights: loads complete in order, so the ids
        // can be used while the weight batch is still in flight.  No branch around the batch
        // (a K step past the wave's last reads its last one; the batch is used only if nb > 0)
        const PrologueIds ld = load_prologue_ids(a);
        setup_weights();
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int s = min(sbase + 4 * u, c1 - 1);
#pragma unroll
            for (int m = 0; m < MT; ++m)
                A0[u][m] = kStreamW ? load_frag_stream(wp[m] + (size_t)s * 512) : load_frag(wp[m] + (size_t)s * 512);
        }
        nact = list_active_from_ids(a, ld, s_list, s_info, s_scr, &id0, &id1);
    } else if (shared_item) {
        setup_weights();
        if (nb > 0) load_w(A0, 0);
    } else if (a.fused && !kDown) {
        nact = list_active_from_ids(a, load_prologue_ids(a), s_list, s_info, s_scr, &id0, &id1);
    } else {
        nact = list_active(a, s_list, s_wsum, s_info);
    }
    // shared groups first: their items can be longer (Fs > F in phase 2), so they
    // start in the first wave of workgroups instead of forming a tail
    if (a.chunked) {
        // group gi (the S shared groups, then the active routed ones) owns
        // ipg x ceil(rows / 16 NT) items, the chunks of one weight slice adjacent
        constexpr int kRows = 16 * NT;
        auto rows_of = [&](int gi) { return gi < a.S ? a.T : max(s_info[gi - a.S].y, 0); };
        const int total = group_prefix(a.S + nact, s_ipre, &s_tot, [&](int gi) {
            return (gi < a.S ? a.ipg_s : a.ipg_r) * ((rows_of(gi) + kRows - 1) / kRows);
        });
        if (item >= total) return;
        int lo = 0, hi = a.S + nact - 1;  // last group with s_ipre[gi] <= item
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_ipre[mid] <= item) lo = mid;
            else hi = mid - 1;
        }
        const int nch = (rows_of(lo) + kRows - 1) / kRows;
        const int local = item - s_ipre[lo];
        sub = local / nch;
        n0 = (local % nch) * kRows;
        if (lo < a.S) {
            g = shared_group(a, lo, sizeof(Elt));
        } else {
            const int4 info = s_info[lo - a.S];
            g = routed_group_of(a, info.x, info.y, info.z, sizeof(Elt));
        }
    } else if (by_slot) {
        // the slot's place in the active list (the lowest, should two experts share a slot)
        for (int p = threadIdx.x; p < nact; p += 256)
            if (s_info[p].z == slot) atomicMin(&s_pos, p);
        __syncthreads();
        const int pos = s_pos;
        if (pos == INT_MAX) return;  // no active expert holds the slot
        const int4 info = s_info[pos];
        g = routed_group_of(a, info.x, info.y, info.z, sizeof(Elt));
        group_rows_from_ids(s_list[pos], a.k, id0, id1, s_gtok, s_wsum);
    } else if (!shared_item) {
        const int i2 = item - a.S * a.ipg_s;
        const int gi = i2 / a.ipg_r;
        if (gi >= nact) return;
        const int4 info = s_info[gi];
        g = routed_group_of(a, info.x, info.y, info.z, sizeof(Elt));
        sub = i2 % a.ipg_r;
        // fused path: the group's token rows from the ids (no perm yet)
        if (a.fused && !kDown) group_rows_from_ids(s_list[gi], a.k, id0, id1, s_gtok, s_wsum);
    }
    if (g.count == 0) return;
    if (!early) {
        setup_weights();
        // the first batch's weights go out before the token rows are looked up
        if (nb > 0) load_w(A0, 0);
    }

    // token operand rows (N side)
    const int ntile = min(NT, (g.count - n0 + 15) / 16);
    const Elt* bp[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        bp[j] = nullptr;
        const int n = n0 + 16 * j + r;
        if (!kDown) {
            const int t = (a.fused && g.routed) ? (n < g.count ? s_gtok[n] : -1) : group_token(a, g, n);
            if (t >= 0) bp[j] = static_cast<const Elt*>(a.x) + (size_t)t * a.H + kq;
        } else if (n < g.count) {
            bp[j] = static_cast<const Elt*>(a.act) + (size_t)(g.rowbase + n) * a.Fa + kq;
        }
    }

    // the K loop for NL token tiles; in the bf16 kernels a group that fills one or two
    // 16-token tiles runs a copy with that many, without the MFMAs of the tiles past its end
    // (separate copies, not a branch in the loop, so that their accumulators never live at
    // once).  The fp32 prefill kernel measured slower with a copy and keeps one loop.
    auto k_loop = [&](auto nl_tag) {
        constexpr int NL = decltype(nl_tag)::value;
        f32x4 acc[MT][NL];
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
            for (int j = 0; j < NL; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};

        auto load_x = [&](F8 (&B)[U][NL], int b) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int s = sbase + 4 * (U * b + u);
#pragma unroll
                for (int j = 0; j < NL; ++j) B[u][j] = (j < ntile && bp[j]) ? load_frag(bp[j] + s * 32) : zero_frag<Elt>();
            }
        };
        auto load = [&](F8 (&A)[U][MT], F8 (&B)[U][NL], int b) {
            load_w(A, b);
            load_x(B, b);
        };
        auto mma = [&](const F8 (&A)[U][MT], const F8 (&B)[U][NL]) {
            // tiles past the group's last token see zero operands: no branch, fewer live registers
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int j = 0; j < NL; ++j)
#pragma unroll
                    for (int m = 0; m < MT; ++m) acc[m][j] = mma_frag(A[u][m], B[u][j], acc[m][j]);
        };
        {
            F8 B0[U][NL], B1[U][NL];
            if (nb > 0) load_x(B0, 0);
            // (rolled: unrolling this loop, which the lambda otherwise invites, slows the fp32 kernel)
#pragma unroll 1
            for (int b = 0; b < nb; b += 2) {
                if (b + 1 < nb) load(A1, B1, b + 1);
                mma(A0, B0);
                if (b + 2 < nb) load(A0, B0, b + 2);
                if (b + 1 < nb) mma(A1, B1);
            }
        }
#pragma unroll 1
        for (int i = nb * U; i < n_my; ++i) {
            const int s = sbase + 4 * i;
            F8 A[MT], B[NL];
#pragma unroll
            for (int m = 0; m < MT; ++m)
                A[m] = kStreamW ? load_frag_stream(wp[m] + (size_t)s * 512) : load_frag(wp[m] + (size_t)s * 512);
#pragma unroll
            for (int j = 0; j < NL; ++j) B[j] = (j < ntile && bp[j]) ? load_frag(bp[j] + s * 32) : zero_frag<Elt>();
#pragma unroll
            for (int j = 0; j < NL; ++j)
#pragma unroll
                for (int m = 0; m < MT; ++m) acc[m][j] = mma_frag(A[m], B[j], acc[m][j]);
        }

#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
            for (int j = 0; j < NL; ++j) s_red[wave][m][j][lane] = acc[m][j];
    };
    if constexpr (sizeof(Elt) == 2 && NT > 1) {
        if (ntile == 1) k_loop(std::integral_constant<int, 1>{});
        else if (NT > 2 && ntile == 2) k_loop(std::integral_constant<int, 2>{});
        else k_loop(std::integral_constant<int, NT>{});
    } else {
        k_loop(std::integral_constant<int, NT>{});
    }
    __syncthreads();

    if (!kDown) {
        // pair gate tile m with up tile m + MH; lane l holds features 4*(l/16)..+3 of token l%16
        for (int task = threadIdx.x; task < MH * NT * kWave; task += 256) {
            const int m = task / (NT * kWave);
            const int j = (task / kWave) % NT;
            const int l = task % kWave;
            const int n = n0 + 16 * j + (l & 15);
            if (j >= ntile || n >= g.count) continue;
            f32x4 gv = s_red[0][m][j][l], uv = s_red[0][m + MH][j][l];
#pragma unroll
            for (int w = 1; w < 4; ++w) {
                gv += s_red[w][m][j][l];
                uv += s_red[w][m + MH][j][l];
            }
            const int f = row0 + 16 * m + 4 * (l >> 4);
            const f32x4 av = {silu(gv.x) * uv.x, silu(gv.y) * uv.y, silu(gv.z) * uv.z, silu(gv.w) * uv.w};
            Elt* dst = static_cast<Elt*>(a.act) + (size_t)(g.rowbase + n) * a.Fa + f;
            if constexpr (sizeof(Elt) == 2) {
                u32x2 packed;
                packed.x = pack_bf16x2(av.x, av.y);
                packed.y = pack_bf16x2(av.z, av.w);
                *reinterpret_cast<u32x2*>(dst) = packed;
            } else {
                *reinterpret_cast<f32x4*>(dst) = av;
            }
        }
    } else {
        for (int task = threadIdx.x; task < MT * NT * kWave; task += 256) {
            const int m = task / (NT * kWave);
            const int j = (task / kWave) % NT;
            const int l = task % kWave;
            const int n = n0 + 16 * j + (l & 15);
            if (j >= ntile || n >= g.count) continue;
            f32x4 v = s_red[0][m][j][l];
#pragma unroll
            for (int w = 1; w < 4; ++w) v += s_red[w][m][j][l];
            const int h = row0 + 16 * m + 4 * (l >> 4);
            float* dst = a.y + (long long)kc * a.y_ks_stride + (size_t)(g.rowbase + n) * a.H + h;
            *reinterpret_cast<f32x4*>(dst) = v;
        }
    }
}

// ---------------------------------------------------------------------------
// tiled kernel (prefill)
// ---------------------------------------------------------------------------
//
// One item = one 256 x 256 output tile of one group: 256 weight rows (phase 1:
// 128 features, their gate and up rows; phase 2: 256 rows of W2) x 256 of the
// group's rows.  Eight waves in 2 (rows) x 4 (tokens), each 128 rows x 64
// tokens = 4 x 2 tiles of v_mfma_f32_32x32x16_bf16 (128 fp32 accumulators per
// lane); a phase-1 wave holds the gate and the up rows of the same 64 features,
// so SwiGLU runs in registers.  Waves 0-3 and 4-7 form two groups with one wave
// of each on every SIMD; wave w has rows w % 2 and token quarter 2 ((w / 2) % 2)
// + w / 4, so a group's end past its first 64 rows keeps both groups busy.  A
// wave whose 64 tokens all lie past the group's end skips its MFMAs.
//
// Schedule (ping-pong): the K loop runs in half-slab phases with a barrier after
// each.  While one wave group reads a slab's operand fragments from LDS (and
// issues its next loads), the other multiplies the slab before, so a SIMD's
// MFMA pipe and the CU's LDS work at once instead of every wave reading after
// the same barrier and then multiplying (on operands already in LDS the
// lockstep loop reaches about two thirds of the MFMA peak, this one about 0.9).
//
// Operands: both are read as 1 KB blocks of the MFMA tile layout (16 rows x 32
// columns; lane l's 16 bytes are row l % 16, columns 8 (l / 16) .. + 7): the
// weights as they are stored, the tokens from a copy that the token gather
// (k_gather_tokens) makes of the resident groups' rows, and phase 2's from the
// activations, which phase 1 writes in that layout.  A CU fills its LDS about
// three times faster from such contiguous blocks than from loads that gather
// 64 bytes from each of 16 row-major token rows.
//
// K runs in 32-wide slabs through a ring of kGStages LDS stages (32 KB each:
// 16 weight blocks, 16 token blocks) filled by direct global->LDS loads: one
// wave instruction moves one 1 KB block, lane l's 16 bytes landing at byte
// 16 l, so every MFMA operand is one conflict-free 16-byte LDS read per lane.
// The loads are issued as inline assembly and waited for by count (the
// compiler cannot see their LDS writes, so it does not make every LDS read wait
// for all of them): each wave issues exactly four per slab and no other
// vector-memory instruction in the K loop, so "slab kt has landed" is "at most
// 4 x (slabs issued after kt) loads outstanding", then a barrier.  The ring is
// the kernel's only LDS: up to kGStages - 1 slabs (128 KB) are in flight, which
// is what the load latency under this traffic asks for.
//
// Items come from a table the token gather writes (one scalar load per item);
// group g owns (weight tiles) x ceil(rows / 256) items, weight tile major.  The
// kernel is persistent, one workgroup per CU: the XCDs get equal contiguous
// ranges of the real items (the hardware deals workgroups to the 8 XCDs
// round-robin), which an XCD's workgroups take in turn, so its 32 CUs start
// each round together on neighbouring tiles of one group and share its weight
// and token panels in their L2.

constexpr int kGM = 256;          // weight rows per item
constexpr int kGN = 256;          // group rows (tokens) per item
constexpr int kGStages = 5;       // LDS ring
constexpr int kGStageBytes = 32 * 1024;

// One item of the tiled kernels (a single 32-byte scalar load).
struct __attribute__((aligned(32))) TileItem {
    int32_t wsel;     // slot of the routed expert (>= 0), or -(s + 1) for shared expert s
    int32_t count;    // rows of the group
    int32_t rowbase;  // first row of the group in the packed row space (y)
    int32_t Fg;       // expert width
    int32_t xblk;     // first row block of the group's token rows in xg
    int32_t ablk;     // first row block of the group's activations
    int32_t wt;       // weight tile
    int32_t n0;       // first group row of the tile
};
// Tile metadata: int32 header[8] (items of phase 1, of phase 2), then
// TileItem phase1[cap1], phase2[cap2].

typedef __attribute__((address_space(3))) uint8_t lds_u8;

// One direct global -> LDS load of 16 bytes per lane: lane l's bytes from g land
// at LDS byte address lds + 16 l (lds is wave-uniform, passed through M0).
__device__ __forceinline__ void lds_load_1k(uint32_t lds, const void* g) {
    asm volatile(
        "s_mov_b32 m0, %0\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %1, off"
        :
        : "s"(lds), "v"(g)
        : "memory", "m0");
}

// Wait until at most N of this wave's vector-memory loads are outstanding and its
// LDS accesses are done, then a workgroup barrier.  The memory clobber keeps
// the compiler's LDS accesses on their side of it.
template <int N>
__device__ __forceinline__ void wait_then_barrier() {
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" : : "n"(N) : "memory");
}

__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}


// Weight tiles of a group of width Fg: phase 1 covers 128 features per tile, phase 2 256 rows of W2.
__device__ __forceinline__ int weight_tiles(const Args& a, int Fg, bool down) {
    return down ? (a.H + kGM - 1) / kGM : (Fg + kGM / 2 - 1) / (kGM / 2);
}

// Writes both phases' item tables: the groups are the active resident routed
// experts (s_list order, with their (segment start, count, slot) in s_info) and
// then the S shared experts; s_bpre holds the routed groups' row-block prefix.
__device__ void write_tile_items(const Args& a, int nact, const int4* s_info, const int* s_bpre, int rb_routed,
                                 int* s_ipre, int* s_tot) {
    const int ng = nact + a.S;
    const int tb16 = (a.T + 15) / 16;
    TileItem* tab = reinterpret_cast<TileItem*>(a.tmeta + 8);
    for (int ph = 0; ph < 2; ++ph) {
        const bool down = ph == 1;
        const int total = group_prefix(ng, s_ipre, s_tot + ph, [&](int gi) {
            const int rows = gi < nact ? max(s_info[gi].y, 0) : a.T;
            const int Fg = gi < nact ? a.F : a.Fs;
            return weight_tiles(a, Fg, down) * ((rows + kGN - 1) / kGN);
        });
        TileItem* out = tab + (down ? a.tcap1 : 0);
        for (int i = threadIdx.x; i < total; i += blockDim.x) {
            int lo = 0, hi = ng - 1;  // last group with s_ipre[g] <= i
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (s_ipre[mid] <= i) lo = mid;
                else hi = mid - 1;
            }
            TileItem it;
            if (lo < nact) {
                const int4 inf = s_info[lo];
                const int P = a.T * a.k;
                const int rb = min(max(inf.x, 0), P);
                it.wsel = inf.z;
                it.count = min(max(inf.y, 0), P - rb);
                it.rowbase = rb;
                it.Fg = a.F;
                it.xblk = s_bpre[lo];
                it.ablk = s_bpre[lo];
            } else {
                const int sh = lo - nact;
                it.wsel = -(sh + 1);
                it.count = a.T;
                it.rowbase = a.T * a.k + sh * a.T;
                it.Fg = a.Fs;
                it.xblk = rb_routed;
                it.ablk = rb_routed + sh * tb16;
            }
            const int ntt = (it.count + kGN - 1) / kGN;
            const int local = i - s_ipre[lo];
            it.wt = local / ntt;
            it.n0 = (local % ntt) * kGN;
            out[i] = it;
        }
        if (threadIdx.x == 0) a.tmeta[ph] = total;
        __syncthreads();  // s_ipre is rewritten for the next phase
    }
}

// The bf16 prefill operands in the MFMA tile layout (16-row x 32-column blocks of
// 1 KB), so that every operand load of the tiled kernel is one contiguous 1 KB
// block.  Row-block space (16 rows per block):
//   xg: routed group gi (active list order) at blocks [bpre[gi], bpre[gi + 1]),
//       its rows in packed order, the rows past the group zero; then, when there
//       are shared experts, the batch's tokens in order at [RB, RB + ceil(T / 16)),
//       RB = bpre[nact];
//   act: the same for the routed groups; shared expert s at RB + s ceil(T / 16).
// Block (rb, c) of a buffer with K columns starts at element (rb K / 32 + c) 512.
// Workgroup 0 also writes the tiled kernels' item tables; the workgroups past
// the row blocks pack the offloaded rows.
__global__ void __launch_bounds__(256) k_gather_tokens(Args a, int blocks_max) {
    __shared__ int s_list[256];
    __shared__ int4 s_info[256];
    __shared__ int s_wsum[8];
    __shared__ int s_bpre[257];
    __shared__ int s_ipre[kGMaxGroups + 1];
    __shared__ int s_tok[16];
    const int pid = blockIdx.x;
    if (pid >= blocks_max) {
        pack_offloaded(a, pid - blocks_max, gridDim.x - blocks_max, 2);
        return;
    }
    const int nact = list_active(a, s_list, s_wsum, s_info);
    const int rb_routed =
        group_prefix(nact, s_bpre, s_wsum + 4, [&](int gi) { return (max(s_info[gi].y, 0) + 15) / 16; });
    if (pid == 0) write_tile_items(a, nact, s_info, s_bpre, rb_routed, s_ipre, s_wsum + 5);
    if (threadIdx.x < 16) {
        const int r = threadIdx.x;
        int t = -1;
        if (pid < rb_routed) {
            int lo = 0, hi = nact - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (s_bpre[mid] <= pid) lo = mid;
                else hi = mid - 1;
            }
            const int4 inf = s_info[lo];
            const Group g = routed_group_of(a, inf.x, inf.y, inf.z, 2);
            t = group_token(a, g, 16 * (pid - s_bpre[lo]) + r);
        } else {
            const int n = 16 * (pid - rb_routed) + r;
            t = (a.S > 0 && n < a.T) ? n : -1;
        }
        s_tok[r] = t;
    }
    __syncthreads();
    if (pid >= rb_routed && (a.S == 0 || pid - rb_routed >= (a.T + 15) / 16)) return;
    // 16-byte piece j of block c: row j % 16, columns 32 c + 8 (j / 16) .. + 7; a batch's
    // loads all go out before its stores (one memory round trip per batch, not per piece)
    const int nc = a.H / 32;
    const uint16_t* x = static_cast<const uint16_t*>(a.x);
    u32x4* dst = reinterpret_cast<u32x4*>(static_cast<uint16_t*>(a.xg) + (size_t)pid * nc * 512);
    constexpr int kBatch = 16;
    for (int base = 0; base < nc * 64; base += 256 * kBatch) {
        u32x4 v[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int idx = base + 256 * u + threadIdx.x;
            const int c = idx >> 6, j = idx & 63;
            const int t = idx < nc * 64 ? s_tok[j & 15] : -1;
            v[u] = u32x4{0u, 0u, 0u, 0u};
            if (t >= 0) v[u] = *reinterpret_cast<const u32x4*>(x + (size_t)t * a.H + 32 * c + 8 * (j >> 4));
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int idx = base + 256 * u + threadIdx.x;
            if (idx < nc * 64) dst[idx] = v[u];
        }
    }
}

// One workgroup per CU (the kernel's LDS admits one), looping over items.  tab: this
// phase's item table, passed on its own and restrict-qualified, so that the compiler knows
// the kernel's stores leave it alone and reads the descriptors through scalar loads (a
// vector load would come with a wait for every outstanding memory operation).
template <bool kDown>
__global__ void __launch_bounds__(512, 1) k_ffn_tiled(Args a, const TileItem* __restrict__ tab) {
    __shared__ __attribute__((aligned(1024))) uint8_t sbuf[kGStages * kGStageBytes];

    // XCD-aware order: XCD x = pid % 8 takes the real items [x per, (x + 1) per), which its
    // workgroups take in turn: the CUs of an XCD start each round together on neighbouring
    // tiles of one group and share its panels in their L2
    const int n_items = a.tmeta[kDown ? 1 : 0];
    const int per = (n_items + 7) / 8;
    const int xcd = blockIdx.x % 8;
    const int xend = min((xcd + 1) * per, n_items);
    const int step = gridDim.x / 8;
    int item = xcd * per + (int)(blockIdx.x / 8);
    TileItem nxt = tab[item < xend ? item : 0];  // the next item's descriptor, loaded one item ahead
    for (; item < xend; item += step) {
        __syncthreads();  // the previous item's epilogue is done with the LDS
        const TileItem it = nxt;
        if (item + step < xend) nxt = tab[item + step];

        const int tid = threadIdx.x, lane = lane_id();
        const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
        const int grp = wave >> 2;  // wave group
        const int wm = wave & 1, wn = 2 * ((wave >> 1) & 1) + grp;
        const int K = kDown ? it.Fg : a.H;
        const int nk = K / 32;  // slabs
        const size_t wsize = (size_t)(kDown ? 1 : 2) * it.Fg * a.H;  // elements of one expert's matrix
        const uint16_t* wbase;
        if (it.wsel >= 0) wbase = static_cast<const uint16_t*>(kDown ? a.w2 : a.w13) + (size_t)it.wsel * wsize;
        else wbase = static_cast<const uint16_t*>(kDown ? a.ws2 : a.ws13) + (size_t)(-it.wsel - 1) * wsize;
        // phase 1: features r0 .. r0 + 127 (gate rows in LDS blocks 0..7, up rows in 8..15);
        // phase 2: rows r0 .. r0 + 255 of W2
        const int r0 = it.wt * (kDown ? kGM : kGM / 2);
        const int rows_out = kDown ? a.H : it.Fg;  // rows (phase 2) or features (phase 1) that exist
        const int n0 = it.n0;

        // 16-row tile of the weight matrix held in LDS weight block b; a block past the
        // matrix reads tile 0 instead (its rows are never stored)
        auto row_tile = [&](int b) -> int {
            if (kDown) {
                const int rt = r0 / 16 + b;
                return 16 * rt < a.H ? rt : 0;
            }
            const int f16 = r0 / 16 + (b & 7);
            if (16 * f16 >= it.Fg) return 0;
            return b < 8 ? f16 : it.Fg / 16 + f16;
        };
        // this wave's loads: weight blocks 2w, 2w + 1 and token blocks 2w, 2w + 1; a token
        // block past the group reads the group's first block instead (never stored)
        const uint16_t* gW0 = wbase + (size_t)row_tile(2 * wave) * nk * 512 + lane * 8;
        const uint16_t* gW1 = wbase + (size_t)row_tile(2 * wave + 1) * nk * 512 + lane * 8;
        const uint16_t* gX[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int nb = n0 / 16 + 2 * wave + i;
            const int blk = (16 * nb < it.count) ? nb : 0;
            if (!kDown)
                gX[i] = static_cast<const uint16_t*>(a.xg) + (size_t)(it.xblk + blk) * (a.H / 32) * 512 + lane * 8;
            else
                gX[i] = static_cast<const uint16_t*>(a.act) + (size_t)(it.ablk + blk) * (a.Fa / 32) * 512 + lane * 8;
        }
        const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_u8*)sbuf;
        auto issue = [&](int kt, int stage) {
            const uint32_t base = lds0 + stage * kGStageBytes;
            lds_load_1k(base + (2 * wave) * 1024, gW0 + (size_t)kt * 512);
            lds_load_1k(base + (2 * wave + 1) * 1024, gW1 + (size_t)kt * 512);
            lds_load_1k(base + (16 + 2 * wave) * 1024, gX[0] + (size_t)kt * 512);
            lds_load_1k(base + (17 + 2 * wave) * 1024, gX[1] + (size_t)kt * 512);
        };

        // operand blocks of this wave: A tile m (32 rows) = LDS weight blocks ab[m], ab[m] + 1;
        // phase 1: m = 0, 1 gate rows, m = 2, 3 the up rows of the same features
        int ab[4];
#pragma unroll
        for (int m = 0; m < 4; ++m)
            ab[m] = kDown ? 8 * wm + 2 * m : (m < 2 ? 4 * wm + 2 * m : 8 + 4 * wm + 2 * (m - 2));
        // B tile jn (32 tokens) = token blocks 16 + 4 wn + 2 jn (+1).  Lane's 16-byte piece of a
        // 32-row (or 32-token) operand at K step s of the slab: block + (l % 32) / 16, piece
        // (l % 16) + 16 (2 s + l / 32)
        const int half = (lane >> 4) & 1;
        const int piece0 = (lane & 15) + 16 * (lane >> 5);
        // a wave whose rows or tokens all lie past the group skips its MFMAs
        const bool live = (n0 + 64 * wn < it.count) && (r0 + (kDown ? 128 : 64) * wm < rows_out);

        f32x16 acc[4][2];
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int jn = 0; jn < 2; ++jn) acc[m][jn] = f32x16{};

        // Phases: in phase 2 kt group 0 reads slab kt's fragments, then issues its loads of
        // slab kt + D, while group 1 multiplies slab kt - 1; in phase 2 kt + 1 group 0
        // multiplies slab kt while group 1 reads it and issues its loads of slab kt + D.  The
        // barrier closing an odd phase 2 kt + 1 also waits for every wave's loads of slab kt + 1.
        // Slab kt + D goes to the stage of slab kt - 1, which both groups have read in phases
        // 2 kt - 2 and 2 kt - 1.  Both groups pass 2 nk + 2 barriers.
        constexpr int D = kGStages - 1;
#pragma unroll
        for (int st = 0; st < D; ++st)
            if (st < nk) issue(st, st);
        auto wait_slab = [&](int n) {  // n: slabs this wave may still have in flight
            __builtin_amdgcn_sched_barrier(0);
            if (n >= 3) wait_then_barrier<12>();
            else if (n == 2) wait_then_barrier<8>();
            else if (n == 1) wait_then_barrier<4>();
            else wait_then_barrier<0>();
            __builtin_amdgcn_sched_barrier(0);
        };
        auto bar_lds = [&]() {  // end of a phase that needs no load to have landed
            __builtin_amdgcn_sched_barrier(0);
            asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" : : : "memory");
            __builtin_amdgcn_sched_barrier(0);
        };
        wait_slab(min(D - 1, nk - 1));  // slab 0
        if (grp == 1) bar_lds();        // phase 0: group 1 has no slab to multiply yet
        int stage = 0;
        for (int kt = 0; kt < nk; ++kt) {
            bf16x8 A[2][4], B[2][2];
            if (live) {
                const uint8_t* sp = sbuf + stage * kGStageBytes;
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const int off = 16 * (piece0 + 32 * ks) + 1024 * half;
#pragma unroll
                    for (int m = 0; m < 4; ++m)
                        A[ks][m] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(sp + ab[m] * 1024 + off));
#pragma unroll
                    for (int jn = 0; jn < 2; ++jn)
                        B[ks][jn] = __builtin_bit_cast(
                            bf16x8, *reinterpret_cast<const u32x4*>(sp + (16 + 4 * wn + 2 * jn) * 1024 + off));
                }
            }
            if (kt + D < nk) issue(kt + D, stage == 0 ? D : stage - 1);
            const int left = min(D - 1, nk - 2 - kt);  // slabs past kt + 1 this wave has in flight
            if (grp == 0) bar_lds();
            else wait_slab(left);
            if (live) {
#pragma unroll
                for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                    for (int m = 0; m < 4; ++m)
#pragma unroll
                        for (int jn = 0; jn < 2; ++jn) acc[m][jn] = mfma32x32x16(A[ks][m], B[ks][jn], acc[m][jn]);
            }
            if (grp == 0) wait_slab(left);
            else bar_lds();
            stage = stage == kGStages - 1 ? 0 : stage + 1;
        }
        if (grp == 0) bar_lds();  // phase 2 nk: group 1 multiplies the last slab
        // Epilogue through the (now idle) LDS ring, so that the global stores are whole
        // rows or whole tile-layout blocks instead of 8-byte pieces of 32 token rows.
        // Lane holds column (token) l % 32 of each 32 x 32 tile, rows 8 (v / 4) + 4 (l / 32) + v % 4.
        __syncthreads();  // every wave is done with the last stage
        if (!kDown) {
            // phase 1: act = silu(gate) * up in bf16, staged in the tile layout of its 16 x 4
            // blocks (token block tb, feature block fb at LDS block 4 tb + fb)
#pragma unroll
            for (int jn = 0; jn < 2; ++jn) {
                const int nl = 64 * wn + 32 * jn + (lane & 31);  // token within the item
#pragma unroll
                for (int m = 0; m < 2; ++m)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int fl = 64 * wm + 32 * m + 8 * q + 4 * (lane >> 5);  // feature within the item
                        const f32x16 gv = acc[m][jn], uv = acc[m + 2][jn];
                        u32x2 packed;
                        packed.x = pack_bf16x2(silu(gv[4 * q]) * uv[4 * q], silu(gv[4 * q + 1]) * uv[4 * q + 1]);
                        packed.y =
                            pack_bf16x2(silu(gv[4 * q + 2]) * uv[4 * q + 2], silu(gv[4 * q + 3]) * uv[4 * q + 3]);
                        const int off = ((nl >> 4) * 4 + (fl >> 5)) * 1024 + 16 * ((nl & 15) + 16 * ((fl & 31) >> 3)) +
                                        2 * (fl & 7);
                        *reinterpret_cast<u32x2*>(sbuf + off) = packed;
                    }
            }
            __syncthreads();
            // 64 blocks of 1 KB; a block goes out if it holds rows of the group and features that exist
            uint16_t* act = static_cast<uint16_t*>(a.act);
            for (int c = tid; c < 64 * 64; c += 512) {
                const int blk = c >> 6, piece = c & 63;
                const int tb = blk >> 2, fb = blk & 3;
                if (n0 + 16 * tb >= it.count || r0 + 32 * fb >= it.Fg) continue;
                const u32x4 v = *reinterpret_cast<const u32x4*>(sbuf + blk * 1024 + 16 * piece);
                *reinterpret_cast<u32x4*>(act + ((size_t)(it.ablk + n0 / 16 + tb) * (a.Fa / 32) + r0 / 32 + fb) * 512 +
                                          8 * piece) = v;
            }
        } else {
            // phase 2: expert outputs in bf16, rounded once (the combine sums them in fp32),
            // staged as 256 token rows of 256 outputs (pitch 264 elements)
            constexpr int kPitch = 264;
            uint16_t* sy = reinterpret_cast<uint16_t*>(sbuf);
#pragma unroll
            for (int jn = 0; jn < 2; ++jn) {
                const int nl = 64 * wn + 32 * jn + (lane & 31);
#pragma unroll
                for (int m = 0; m < 4; ++m)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int hl = 128 * wm + 32 * m + 8 * q + 4 * (lane >> 5);
                        const f32x16 v = acc[m][jn];
                        u32x2 packed;
                        packed.x = pack_bf16x2(v[4 * q], v[4 * q + 1]);
                        packed.y = pack_bf16x2(v[4 * q + 2], v[4 * q + 3]);
                        *reinterpret_cast<u32x2*>(sy + nl * kPitch + hl) = packed;
                    }
            }
            __syncthreads();
            // 256 rows x 32 pieces of 16 bytes; rows of the group, outputs that exist
            for (int c = tid; c < 256 * 32; c += 512) {
                const int nl = c >> 5, piece = c & 31;
                const int h = r0 + 8 * piece;
                if (n0 + nl >= it.count || h >= a.H) continue;
                const u32x4 v = *reinterpret_cast<const u32x4*>(sy + nl * kPitch + 8 * piece);
                *reinterpret_cast<u32x4*>(a.y16 + (size_t)(it.rowbase + n0 + nl) * a.H + h) = v;
            }
        }
    }
}

// y_out[p] = sum_c y[c][p] for resident packed rows p < n_res and all shared rows
// (kInBf16: a single chunk of bf16 rows, widened).
template <bool kInBf16>
__global__ void __launch_bounds__(256) k_reduce_splits(int T, int H, int E, int k, int S, int slots,
                                                       const int32_t* __restrict__ counts,
                                                       const int32_t* __restrict__ expert_slot,
                                                       const void* __restrict__ y_in, int ks, long long stride,
                                                       float* __restrict__ y_out) {
    __shared__ int s_nres;
    if (threadIdx.x == 0) {
        int n = 0;
        for (int e = 0; e < E; ++e)
            if (is_resident(expert_slot[e], slots)) n += counts[e] > 0 ? counts[e] : 0;
        s_nres = n;
    }
    __syncthreads();
    const int P = T * k, rows = P + S * T;
    const int row = blockIdx.x;
    if (row >= rows || (row < P && row >= s_nres)) return;
    if constexpr (kInBf16) {
        const uint16_t* y = static_cast<const uint16_t*>(y_in);
        for (int h = threadIdx.x * 4; h < H; h += 1024)
            *reinterpret_cast<f32x4*>(y_out + (size_t)row * H + h) =
                bf16x4_to_f32(*reinterpret_cast<const u32x2*>(y + (size_t)row * H + h));
        return;
    }
    const float* y = static_cast<const float*>(y_in);
    for (int h = threadIdx.x * 4; h < H; h += 1024) {
        constexpr int kMax = 16;  // same order as the combine: chunk 0, then 1, ...
        f32x4 p[kMax];
#pragma unroll
        for (int c = 0; c < kMax; ++c)
            if (c < ks) p[c] = *reinterpret_cast<const f32x4*>(y + c * stride + (size_t)row * H + h);
        f32x4 v = p[0];
#pragma unroll
        for (int c = 1; c < kMax; ++c)
            if (c < ks) v += p[c];
        *reinterpret_cast<f32x4*>(y_out + (size_t)row * H + h) = v;
    }
}

int max_routed_groups(const Shape& s) {
    int m = s.E < s.slots ? s.E : s.slots;
    const int pairs = s.T * s.k;
    return m < pairs ? m : pairs;
}

bool use_stream(const Shape& s) { return s.T <= 64; }

template <typename Elt, bool kDown, bool kStreamW>
void launch_stream_w(int nt, int grid, const Args& a, hipStream_t st) {
    switch (nt) {
        case 1: hipLaunchKernelGGL((k_ffn_stream<Elt, 1, kDown, kStreamW>), dim3(grid), dim3(256), 0, st, a); break;
        case 2: hipLaunchKernelGGL((k_ffn_stream<Elt, 2, kDown, kStreamW>), dim3(grid), dim3(256), 0, st, a); break;
        case 3: hipLaunchKernelGGL((k_ffn_stream<Elt, 3, kDown, kStreamW>), dim3(grid), dim3(256), 0, st, a); break;
        default: hipLaunchKernelGGL((k_ffn_stream<Elt, 4, kDown, kStreamW>), dim3(grid), dim3(256), 0, st, a); break;
    }
}

template <typename Elt, bool kDown>
void launch_stream(int nt, bool stream_w, int grid, const Args& a, hipStream_t st) {
    if (stream_w) launch_stream_w<Elt, kDown, true>(nt, grid, a, st);
    else launch_stream_w<Elt, kDown, false>(nt, grid, a, st);
}

// Non-temporal weight loads when the weights one call can touch (every slot and
// shared expert) exceed a quarter of the 256 MB MALL: then they cannot stay in
// the caches from one call to the next anyway.
bool stream_weights(const Shape& s) {
    const long long b = s.bf16 ? 2 : 4;
    const long long bytes = 3ll * s.H * ((long long)s.slots * s.F + (long long)s.S * s.Fs) * b;
    return bytes > (64ll << 20);
}

}  // namespace

bool ffn_packs_offloaded(const Shape& s) { return use_stream(s) || s.bf16; }

bool ffn_fuses_repack(const Shape& s) { return use_stream(s) && s.T > 0; }

namespace {
// bf16 prefill: row blocks of the routed groups padded to 16 rows (at most 15 pad
// rows per group) and of the batch in order
long long tiled_routed_rows(const Shape& s) {
    return (long long)s.T * s.k + 15ll * max_routed_groups(s);
}
long long tiled_t16(const Shape& s) { return (s.T + 15) / 16 * 16ll; }
bool use_tiled(const Shape& s) { return s.bf16 && !use_stream(s); }

// Worst-case items of a tiled phase: the routed groups have at most ceil(P / 256)
// full 256-row tiles plus one partial tile each
long long tiled_items(const Shape& s, bool down) {
    const long long P = (long long)s.T * s.k;
    const long long G = max_routed_groups(s);
    const long long rt = G == 0 ? 0 : (P + kGN - 1) / kGN + G;
    const long long tps = (s.T + kGN - 1) / kGN;
    if (down) return (rt + (long long)s.S * tps) * ((s.H + kGM - 1) / kGM);
    const long long wt_r = (s.F + kGM / 2 - 1) / (kGM / 2), wt_s = s.S > 0 ? (s.Fs + kGM / 2 - 1) / (kGM / 2) : 0;
    return rt * wt_r + (long long)s.S * tps * wt_s;
}

Args make_args(const Shape& s, const FfnArgs& fa) {
    Args a;
    a.T = s.T; a.H = s.H; a.E = s.E; a.F = s.F; a.k = s.k; a.S = s.S; a.Fs = s.Fs; a.slots = s.slots;
    a.x = fa.x; a.perm = fa.perm; a.counts = fa.counts; a.seg_start = fa.seg_start; a.expert_slot = fa.expert_slot;
    a.w13 = fa.w13; a.w2 = fa.w2; a.ws13 = fa.ws13; a.ws2 = fa.ws2;
    a.act = fa.act; a.Fa = fa.Fa; a.y = fa.y; a.ks = fa.ks; a.y_ks_stride = fa.y_ks_stride;
    a.max_routed = max_routed_groups(s);
    a.ipg_r = a.ipg_s = 0;
    a.chunked = 0;
    a.topk_w = fa.topk_w;
    a.n_res = fa.n_res;
    a.off_rows = fa.off_rows;
    a.off_w = fa.off_w;
    a.xg = fa.xg;
    a.tmeta = fa.tmeta;
    a.tcap1 = use_tiled(s) ? (int)tiled_items(s, false) : 0;
    a.y16 = static_cast<uint16_t*>(fa.y16);
    a.fused = fa.topk_idx != nullptr;
    // every slot can hold an active expert: the fused phase 1 maps routed items to slots
    a.slot_items = (s.T * s.k >= s.slots && s.E >= s.slots) ? 1 : 0;
    a.topk_idx = fa.topk_idx;
    a.rp_counts = fa.rp_counts;
    a.rp_seg_start = fa.rp_seg_start;
    a.rp_perm = fa.rp_perm;
    a.rp_inv_perm = fa.rp_inv_perm;
    a.rp_n_res = fa.rp_n_res;
    return a;
}
}  // namespace

long long ffn_act_rows(const Shape& s) {
    if (use_tiled(s)) return tiled_routed_rows(s) + (long long)s.S * tiled_t16(s);
    return (long long)s.T * s.k + (long long)s.S * s.T;
}

long long ffn_gather_rows(const Shape& s) {
    if (!use_tiled(s)) return 0;
    return tiled_routed_rows(s) + (s.S > 0 ? tiled_t16(s) : 0);
}

size_t ffn_tile_meta_bytes(const Shape& s) {
    if (!use_tiled(s)) return 0;
    return 32 + sizeof(TileItem) * (size_t)(tiled_items(s, false) + tiled_items(s, true));
}

hipError_t launch_gather_tokens(const Shape& s, const FfnArgs& fa, hipStream_t st) {
    if (s.T == 0 || !use_tiled(s)) return hipSuccess;
    const Args a = make_args(s, fa);
    const long long blocks = ffn_gather_rows(s) / 16;
    const int P = s.T * s.k;
    const int n_pack = (fa.off_rows || fa.off_w) ? (P < 256 ? P : 256) : 0;
    hipLaunchKernelGGL(k_gather_tokens, dim3((unsigned)(blocks + n_pack)), dim3(256), 0, st, a, (int)blocks);
    return hipGetLastError();
}

int ffn_down_splits(const Shape& s) {
    if (!use_stream(s)) return 1;
    // Phase-2 work items: (groups) x (H / rows) x ks, each streaming `rows` rows
    // (16 per weight tile) of one K chunk.  Smallest ks (a power of two <= 16) such that
    //  * there are >= 512 workgroups (two per CU), and
    //  * the longest workgroup streams at most 1/400 of the phase's weights: one
    //    workgroup streams at about 1/200 of the chip's HBM rate, so with a 2x
    //    margin it then ends before the phase does, instead of forming its tail
    //    (a shared expert wider than the routed ones, or few wide experts);
    // while every wave keeps >= 8 K steps of 32.
    const long long groups_r = max_routed_groups(s);
    const long long groups = groups_r + s.S;
    if (groups == 0) return 1;
    int steps = s.F / 32;
    if (s.S > 0 && s.Fs / 32 < steps) steps = s.Fs / 32;
    const long long kmax = (s.S > 0 && s.Fs > s.F) ? s.Fs : s.F;
    const long long weights = (groups_r * s.F + (long long)s.S * s.Fs) * s.H;  // elements, worst case
    const long long rows = 16 * stream_mt((s.T + 15) / 16);
    auto balanced = [&](int ks) { return groups * (s.H / rows) * ks >= 512 && rows * kmax / ks * 400 <= weights; };
    int ks = 1;
    while (ks < 16 && !balanced(ks) && steps / (ks * 2) >= 16) ks *= 2;
    return ks;
}

hipError_t launch_grouped_ffn(const Shape& s, const FfnArgs& fa, hipStream_t st, hipEvent_t between) {
    if (s.T == 0) return hipSuccess;
    auto mark = [&]() -> hipError_t {
        hipError_t e = hipGetLastError();
        if (e == hipSuccess && between) e = hipEventRecord(between, st);
        return e;
    };
    Args a = make_args(s, fa);
    if (!s.bf16 && !use_stream(s)) {
        // fp32 prefill: the stream kernel over chunks of 64 rows; a workgroup per
        // worst-case item: the routed groups hold at most ceil(P / 64) full chunks
        // plus one partial chunk each
        a.chunked = 1;
        const long long chunks_r = a.max_routed == 0 ? 0 : ((long long)s.T * s.k + 63) / 64 + a.max_routed;
        const long long chunks_s = (long long)s.S * ((s.T + 63) / 64);
        a.ipg_r = s.F / 32;
        a.ipg_s = s.S > 0 ? s.Fs / 32 : 1;
        long long grid = a.ipg_r * chunks_r + a.ipg_s * chunks_s;
        if (grid > 0)
            hipLaunchKernelGGL((k_ffn_stream<float, 4, false, false>), dim3((unsigned)grid), dim3(256), 0, st, a);
        if (hipError_t e = mark(); e != hipSuccess) return e;
        a.ipg_r = a.ipg_s = s.H / 64;
        grid = a.ipg_r * (chunks_r + chunks_s);
        if (grid > 0)
            hipLaunchKernelGGL((k_ffn_stream<float, 4, true, false>), dim3((unsigned)grid), dim3(256), 0, st, a);
        return hipGetLastError();
    }
    if (use_stream(s)) {
        const int nt = (s.T + 15) / 16;
        const bool sw = stream_weights(s);
        // phase 1: 32 features per workgroup
        const int mt = stream_mt(nt);
        a.ipg_r = s.F / (8 * mt);
        a.ipg_s = s.S > 0 ? s.Fs / (8 * mt) : 1;
        const int P = s.T * s.k;
        const int n_pack = (fa.off_rows || fa.off_w) ? (P < 64 ? P : 64) : 0;  // pack workgroups (P >= 1)
        // phase 1, then (fused) the repack workgroup, or the pack workgroups
        int grid = a.max_routed * a.ipg_r + s.S * a.ipg_s + (a.fused ? 1 : n_pack);
        if (grid > 0) {
            if (s.bf16) launch_stream<uint16_t, false>(nt, sw, grid, a, st);
            else launch_stream<float, false>(nt, sw, grid, a, st);
        }
        if (hipError_t e = mark(); e != hipSuccess) return e;
        // phase 2: 64 output rows x one K chunk per workgroup; (fused) then the pack
        // workgroups, which read the perm and n_res that phase 1 wrote
        a.ipg_r = (s.H / (16 * mt)) * a.ks;
        a.ipg_s = (s.H / (16 * mt)) * a.ks;
        grid = a.max_routed * a.ipg_r + s.S * a.ipg_s + (a.fused ? n_pack : 0);
        if (grid > 0) {
            if (s.bf16) launch_stream<uint16_t, true>(nt, sw, grid, a, st);
            else launch_stream<float, true>(nt, sw, grid, a, st);
        }
        return hipGetLastError();
    }
    // tiled: one workgroup per CU, each taking its XCD's items from the table the token
    // gather wrote in turn; the offloaded rows were packed by the token gather
    int dev = 0, cus = 0;
    if (hipError_t e = hipGetDevice(&dev); e != hipSuccess) return e;
    if (hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev); e != hipSuccess)
        return e;
    const long long wgs = cus < 8 ? 8 : cus / 8 * 8;
    auto tiled_grid = [&](long long items) { return items < wgs ? (items + 7) / 8 * 8 : wgs; };
    {
        const long long grid = tiled_grid(tiled_items(s, false));
        if (grid > 0)
            hipLaunchKernelGGL((k_ffn_tiled<false>), dim3((unsigned)grid), dim3(512), 0, st, a,
                               reinterpret_cast<const TileItem*>(a.tmeta + 8));
    }
    if (hipError_t e = mark(); e != hipSuccess) return e;
    {
        const long long grid = tiled_grid(tiled_items(s, true));
        if (grid > 0)
            hipLaunchKernelGGL((k_ffn_tiled<true>), dim3((unsigned)grid), dim3(512), 0, st, a,
                               reinterpret_cast<const TileItem*>(a.tmeta + 8) + a.tcap1);
    }
    return hipGetLastError();
}

hipError_t launch_reduce_splits(const Shape& s, const int32_t* counts, const int32_t* expert_slot, const void* y,
                                bool y_bf16, int ks, long long y_ks_stride, float* y_out, hipStream_t st) {
    const int rows = s.T * s.k + s.S * s.T;
    if (rows == 0) return hipSuccess;
    if (y_bf16)
        hipLaunchKernelGGL(k_reduce_splits<true>, dim3(rows), dim3(256), 0, st, s.T, s.H, s.E, s.k, s.S, s.slots,
                           counts, expert_slot, y, 1, y_ks_stride, y_out);
    else
        hipLaunchKernelGGL(k_reduce_splits<false>, dim3(rows), dim3(256), 0, st, s.T, s.H, s.E, s.k, s.S, s.slots,
                           counts, expert_slot, y, ks, y_ks_stride, y_out);
    return hipGetLastError();
}

bool ffn_y_bf16(const Shape& s) { return use_tiled(s); }

size_t ffn_y_bytes(const Shape& s) {
    const long long rows = (long long)s.T * s.k + (long long)s.S * s.T;
    if (ffn_y_bf16(s)) return (size_t)rows * s.H * 2;
    return (size_t)ffn_down_splits(s) * rows * s.H * 4;
}

}  // namespace saem
