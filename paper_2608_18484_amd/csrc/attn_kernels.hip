// Attention-side kernels of the SparsePR operator for gfx950:
//  * renormalised hard-drop block-sparse attention over the routed cells
//    (Sec. 3 eq. hard_drop; Sec. 4.3), bf16 MFMA with fp32 accumulation, or
//    an fp32 VALU variant;
//  * exact probe rows against all keys (Sec. 4.3; App. A.2 eq.
//    app_probe_residual), split over keys and merged by log-sum-exp;
//  * the probe-fitted residual fit, correction and restore are launched from
//    here and live in fit_kernels.hip.
//
// Layout of the bf16 attention kernel.  A block of 128 threads (2 waves)
// owns up to 64 query rows of one query group; each wave owns 32 of them.
// The scores are formed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16
// (A = 32 keys x 16 dims from LDS, B = 16 dims x 32 queries held in
// registers), so every lane holds scores of ONE query and the online softmax
// needs a single cross-lane exchange (lanes l and l+32).  The probabilities
// stay in registers and feed O^T = V^T P^T directly as the B operand; V stays
// row-major in LDS and its A operand V^T comes from transposing LDS reads
// (ds_read_b64_tr_b16), the keys of each 16-key chunk taken in the order of
// the accumulator layout.
// K/V rows are gathered on load through the group-major permutation, so the
// routed K/V groups are contiguous key ranges without a physical copy.
#include <hip/hip_runtime.h>
#include <math.h>

#include <type_traits>

#include "device_utils.hpp"
#include "sparsepr_internal.hpp"

namespace sparsepr {

enum { MODE_SPARSE = 0, MODE_PROBE = 1, MODE_DENSE = 2 };

struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  void* out;          // MODE_DENSE: user output tensor
  float* osp;         // MODE_SPARSE: [BH][N][D] fp32
  float* part;        // MODE_PROBE: [BH][M][nsplit][D+2]
  const int4* chunks;
  const int32_t* nchunks;
  const int32_t* permq;
  const int32_t* offq;
  const int32_t* permk;
  const int2* rng;
  const int32_t* rng_cnt;
  const int32_t* probes;
  const int32_t* nprobes;
  const uint16_t* kperm;
  const uint16_t* vperm;
  // MODE_SPARSE key segment: only keys at group-major positions in
  // [seg_lo, seg_hi) are processed; (O, m, l) carry over between segments
  float* mlst;
  int seg_lo, seg_hi, seg_first, seg_last;
  int heads_per_xcd;  // MODE_SPARSE block order (see k_attn_mfma)
};

// Where the rows and keys of one block come from.
struct Work1 {
  int nrows;      // valid query rows (<= 64)
  int nkeys;      // keys in the flat key list
  int k0;         // MODE_PROBE/DENSE: first key row
  int a;          // MODE_SPARSE: query group
  int rbase;      // MODE_SPARSE: first permutation slot of the rows
  int split;      // MODE_PROBE: split index
  int tile;       // MODE_PROBE/DENSE: row tile
};

template <int MODE>
__device__ __forceinline__ bool get_work(const Geom& g, const AttnArgs& A, int bh, Work1& w) {
  if (MODE == MODE_SPARSE) {
    const int cx = blockIdx.x;
    if (cx >= A.nchunks[bh]) return false;
    const int4 c = A.chunks[(size_t)bh * g.nchunk_max + cx];
    w.a = c.x;
    w.rbase = A.offq[(size_t)bh * (g.CQt + 1) + c.x] + c.y;
    w.nrows = c.z;
    w.nkeys = c.w;
    w.k0 = 0;
    return w.nrows > 0 && w.nkeys > 0;
  } else if (MODE == MODE_PROBE) {
    const int np = A.nprobes[bh];
    w.tile = blockIdx.x;
    w.split = blockIdx.y;
    if (w.tile * 64 >= np) return false;
    w.nrows = min(64, np - w.tile * 64);
    w.k0 = w.split * kProbeSplit;
    w.nkeys = min(g.N - w.k0, kProbeSplit);
    return w.nkeys > 0;
  } else {
    w.tile = blockIdx.x;
    w.nrows = min(64, g.N - w.tile * 64);
    w.k0 = 0;
    w.nkeys = g.N;
    return w.nrows > 0;
  }
}

template <int MODE>
__device__ __forceinline__ int row_of(const Geom& g, const AttnArgs& A, int bh, const Work1& w,
                                      int r) {
  if (MODE == MODE_SPARSE) return A.permq[(size_t)bh * g.N + w.rbase + r];
  if (MODE == MODE_PROBE) return A.probes[(size_t)bh * g.M + w.tile * 64 + r];
  return w.tile * 64 + r;
}

// Source row of flat key f (f < nkeys).  MODE_SPARSE walks the routed ranges
// with a per-thread cursor that only moves forward.
struct KeyCursor {
  int j, cum;
};

template <int MODE>
__device__ __forceinline__ int key_row(const Geom& g, const AttnArgs& A, int bh, const Work1& w,
                                       int f, KeyCursor& cur, const int2* rg, int nr) {
  if (MODE != MODE_SPARSE) return w.k0 + f;
  while (cur.j < nr && f >= cur.cum + rg[cur.j].y) {
    cur.cum += rg[cur.j].y;
    ++cur.j;
  }
  return A.permk[(size_t)bh * g.N + rg[cur.j].x + (f - cur.cum)];
}

// Bank swizzle of the 16-byte chunks of a K/V tile row in LDS: chunk c of
// key r sits at position c ^ swz(r).  A 16-lane phase of a 128-bit read (the
// K operand) takes one chunk of 16 consecutive keys, and one of a transposing
// read takes two neighbouring chunks of 4 consecutive keys (two phases: four
// chunks).  With 256-byte rows (D = 128) a row spans the 64 banks once, so
// swz is a bijection of 16 consecutive keys onto the 16 chunk positions whose
// bits 2-3 differ within every aligned group of 4 keys: both reads hit
// distinct banks.  With 128-byte rows (D = 64) two keys share a bank row and
// the 3-bit form is used.
template <int D>
__device__ __forceinline__ int kv_swz(int r) {
  if (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  return ((r & 3) << 1) | ((r >> 2) & 1);
}

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

// LDS transposing read of four 16-bit values.  In every group of 16 lanes,
// lane j receives element j%4 of the 8-byte rows addressed by lanes
// j/4, j/4+4, j/4+8, j/4+12 of its group.
__device__ __forceinline__ v4i16 lds_read_tr16(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_v4i16*)(__attribute__((address_space(3))) uint16_t*)(p));
}

// Direct global->LDS copy of 16 bytes per lane: lane l's bytes land at
// lds_base + 16*l (lds_base must be the same for the whole wave).  Issued as
// inline assembly so that the compiler adds no waits for it; callers order it
// with explicit s_waitcnt vmcnt.  Nothing else in these kernels uses M0.
__device__ __forceinline__ void g2lds16(const void* src, const void* lds_base) {
  const uint32_t lds = __builtin_amdgcn_readfirstlane(
      (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)lds_base);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(lds)
               : "memory");
}

// The same copy addressed as a uniform 64-bit base (SGPRs) plus a 32-bit
// per-lane byte offset; `m0v` is the wave-uniform LDS destination.
__device__ __forceinline__ void g2lds16s(const void* sbase, uint32_t voff, uint32_t m0v) {
  // readfirstlane returns a signed int: widen through uint32_t so the low
  // half of the address is zero-extended, never sign-extended
  const uint64_t b = (uint64_t)(size_t)sbase;
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  const uint64_t sb = ((uint64_t)hi << 32) | (uint64_t)lo;
  const uint32_t m0u = (uint32_t)__builtin_amdgcn_readfirstlane(m0v);
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 offset:0"
               :
               : "v"(voff), "s"(sb), "s"(m0u)
               : "memory");
}

// Combine a value with the one held by lane l ^ 32 (the other half of the
// same query's keys) through v_permlane32_swap: swapping a register with
// itself leaves, in each lane, its own value in one result and its partner's
// in the other, so max3 / the sum of both results combine the pair.
__device__ __forceinline__ float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Block-sparse flash attention, bf16 MFMA, fp32 accumulation.
//  * 128 threads = 2 waves; a block owns up to 64 query rows (32 per wave)
//    that share one key list: the routed ranges of their query group in the
//    group-major K/V copy (MODE_SPARSE), or a contiguous slice of the original
//    K/V rows (MODE_PROBE, MODE_DENSE).
//  * 32-key tiles in LDS filled by direct global->LDS 16-byte loads: one K
//    buffer, refilled with the next tile once every wave has read its score
//    operands, and two V buffers, the next tile's V loading while the current
//    one is computed; the key positions of a tile are computed two tiles
//    ahead into a ring of three slots.  The 26 KB of LDS and at most 168
//    registers per lane leave room for six blocks per CU (three waves per
//    SIMD), which hide each other's latencies better than four.
//  * S^T = K Q^T and O^T += V^T P^T with v_mfma_f32_32x32x16_bf16; V^T
//    fragments come from the row-major V tile through transposing LDS reads.
//  * Online softmax in base 2 with lazy rescaling: the running maximum only
//    moves (and O, l are rescaled) when a tile's maximum exceeds it by 2^8.
template <int D, int MODE>
__global__ __launch_bounds__(128) __attribute__((amdgpu_waves_per_eu(3, 3))) void k_attn_mfma(Geom g, AttnArgs A) {
  constexpr int KT = 32;
  constexpr int CH = D / 8;                    // 16-byte chunks per row
  constexpr int NKS = D / 16;                  // k-steps of Q K^T
  constexpr int NDB = D / 32;                  // 32-wide blocks of O^T
  constexpr int LPT = KT * CH / 128;           // 16-byte loads per thread per tensor per tile
  constexpr int MAXR = 128;                    // routed ranges of the segment staged in LDS
  // tiles[0] = K (one buffer), tiles[1..2] = V (double-buffered)
  __shared__ __attribute__((aligned(1024))) uint16_t tiles[3][KT * D];
  __shared__ int spos[3][KT];
  __shared__ int2 srng[MODE == MODE_SPARSE ? MAXR : 1];

  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  Work1 w;
  int bh;
  const uint16_t* Kp;
  const uint16_t* Vp;
  if (MODE == MODE_SPARSE) {
    // XCD-aware order: hardware block b runs on XCD b % 8.
    //  * heads_per_xcd (head count a multiple of 8): grid (8 * nchunk_max,
    //    BH / 8); XCD x runs every chunk of heads x, x + 8, ... in turn, so
    //    its L2 only ever holds one head's K/V segment and all of that
    //    head's query groups reuse it.
    //  * otherwise: grid (8 * ceil(nchunk_max / 8), BH); XCD x takes the
    //    contiguous slice [x*per, (x+1)*per) of each head's chunks.
    int cx;
    if (A.heads_per_xcd) {
      bh = blockIdx.y * 8 + (blockIdx.x & 7);
      cx = blockIdx.x >> 3;
      if (cx >= A.nchunks[bh]) return;
    } else {
      bh = blockIdx.y;
      const int nch = A.nchunks[bh];
      const int per = (nch + 7) / 8;
      const int x = blockIdx.x & 7, y = blockIdx.x >> 3;
      cx = x * per + y;
      if (y >= per || cx >= nch) return;
    }
    const int4 c = A.chunks[(size_t)bh * g.nchunk_max + cx];
    w.a = c.x;
    w.rbase = A.offq[(size_t)bh * (g.CQt + 1) + c.x] + c.y;
    w.nrows = c.z;
    w.nkeys = c.w;
    w.k0 = 0;
    if (w.nrows <= 0 || w.nkeys <= 0) return;  // every routed query group has keys
    Kp = A.kperm + (size_t)bh * g.N * D;
    Vp = A.vperm + (size_t)bh * g.N * D;
  } else {
    bh = (MODE == MODE_PROBE) ? blockIdx.z : blockIdx.y;
    if (!get_work<MODE>(g, A, bh, w)) return;
    const int64_t base = kv_base(g, bh);
    Kp = (const uint16_t*)A.k + base;
    Vp = (const uint16_t*)A.v + base;
  }
  const int64_t ksn = (MODE == MODE_SPARSE) ? D : g.sn;  // row stride of Kp/Vp
  const int64_t qbase = q_base(g, bh, g.gq);  // also the output's, in MODE_DENSE
  const uint16_t* Qp = (const uint16_t*)A.q + qbase;

  // query row of this lane and its B operands
  const int qr = wv * 32 + n;
  const bool qvalid = qr < w.nrows;
  const int qrow = qvalid ? row_of<MODE>(g, A, bh, w, qr) : 0;
  bf16x8 qreg[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    uint4 u = make_uint4(0, 0, 0, 0);
    if (qvalid) u = *(const uint4*)(Qp + (int64_t)qrow * g.sn + ks * 16 + h * 8);
    qreg[ks] = __builtin_bit_cast(bf16x8, u);
  }
  const bool wave_active = wv * 32 < w.nrows;

  // routed ranges of the query group (positions in the group-major K/V);
  // never read through generic pointers (flat accesses would make the
  // compiler wait for the in-flight tile loads).  Only the ranges meeting the
  // key segment [seg_lo, seg_hi) are walked, each clipped to it: ranges are
  // sorted and disjoint, so they are the run [j0, j0 + nseg) and their
  // clipped lengths sum to this launch's keys; the first MAXR of the run are
  // staged in LDS.
  typedef const __attribute__((address_space(1))) int* gptr_int;
  gptr_int grng = nullptr;
  int nr = 0, j0 = 0, nseg = 0;
  __shared__ int sred[2][3];
  if (MODE == MODE_SPARSE) {
    grng = (gptr_int)(A.rng + ((size_t)bh * g.CQt + w.a) * g.CKt);
    nr = A.rng_cnt[(size_t)bh * g.CQt + w.a];
    int below = 0, before_end = 0, keys = 0;
    for (int i = tid; i < nr; i += 128) {
      const int2 r = make_int2(grng[2 * i], grng[2 * i + 1]);
      below += (r.x + r.y <= A.seg_lo);
      before_end += (r.x < A.seg_hi);
      keys += max(min(r.x + r.y, A.seg_hi) - max(r.x, A.seg_lo), 0);
    }
    below = wave_sum_i(below);
    before_end = wave_sum_i(before_end);
    keys = wave_sum_i(keys);
    if (lane == 0) {
      sred[wv][0] = below;
      sred[wv][1] = before_end;
      sred[wv][2] = keys;
    }
    __syncthreads();
    j0 = sred[0][0] + sred[1][0];
    nseg = sred[0][1] + sred[1][1] - j0;
    w.nkeys = sred[0][2] + sred[1][2];
    for (int i = tid; i < min(nseg, MAXR); i += 128)
      srng[i] = make_int2(grng[2 * (j0 + i)], grng[2 * (j0 + i) + 1]);
    __syncthreads();
  }
  auto range_at = [&](int j) -> int2 {  // clipped range j of the segment's run
    const int jj = j0 + j;
    const int2 r = (j < MAXR) ? srng[j] : make_int2(grng[2 * jj], grng[2 * jj + 1]);
    const int lo = max(r.x, A.seg_lo), hi = min(r.x + r.y, A.seg_hi);
    return make_int2(lo, hi - lo);
  };
  const int safe_pos = (MODE == MODE_SPARSE) ? (nseg > 0 ? range_at(0).x : 0) : w.k0;
  // Each of lanes 0-31 of wave 0 walks the ranges for key tid of every tile
  // with a cursor that only moves forward.  The cursor's range and the one
  // after it are kept in registers, so a tile costs no dependent LDS read
  // unless its key crosses two range boundaries; the read of the new next
  // range is only waited for at the following crossing.
  KeyCursor cur{0, 0};
  int2 cr = make_int2(0, 0), nx = make_int2(0, 0);
  if (MODE == MODE_SPARSE && tid < KT && nseg > 0) {
    cr = range_at(0);
    nx = nseg > 1 ? range_at(1) : make_int2(0, 0x7fffffff);
  }
  auto fill_pos = [&](int tt) {  // key positions of tile tt -> ring slot tt % 3
    if (tid < KT) {
      const int f = tt * KT + tid;
      int pos = safe_pos;
      if (f < w.nkeys) {
        if (MODE == MODE_SPARSE) {
          while (f >= cur.cum + cr.y) {  // f < nkeys: the run ends after f
            cur.cum += cr.y;
            ++cur.j;
            cr = nx;
            nx = cur.j + 1 < nseg ? range_at(cur.j + 1) : make_int2(0, 0x7fffffff);
          }
          pos = cr.x + (f - cur.cum);
        } else {
          pos = w.k0 + f;
        }
      }
      spos[tt % 3][tid] = pos;
    }
  };
  // LDS byte address of tiles[0] (uniform); the K buffer is there, V
  // buffer b at +(1+b)*KT*D*2
  const uint32_t lds_tiles = __builtin_amdgcn_readfirstlane(
      (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)&tiles[0][0]);
  const uint32_t row_bytes = (uint32_t)(ksn * 2);
  // the copies of tile tt of one tensor into the buffer at dst
  auto issue = [&](int tt, const uint16_t* src, uint32_t dst) {
    // all positions first (one LDS wait), then the copies
    uint32_t voff[LPT];
#pragma unroll
    for (int u = 0; u < LPT; ++u) {
      const int inst = wv * LPT + u;
      const int s = inst * 64 + lane;
      const int key = s / CH, p = s % CH;
      const int c8 = p ^ kv_swz<D>(key);
      voff[u] = (uint32_t)spos[tt % 3][key] * row_bytes + (uint32_t)(c8 * 16);
    }
#pragma unroll
    for (int u = 0; u < LPT; ++u) g2lds16s(src, voff[u], dst + (uint32_t)((wv * LPT + u) * 1024));
  };
  const uint32_t kdst = lds_tiles;
  auto vdst = [&](int b) { return lds_tiles + (uint32_t)((1 + b) * KT * D * 2); };

  const float sl2 = 1.4426950408889634f / sqrtf((float)D);
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 O[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) O[db][i] = 0.f;
  if (MODE == MODE_SPARSE && !A.seg_first && qvalid) {
    // resume the running state left by the previous key segment
    const float* src = A.osp + ((size_t)bh * g.N + qrow) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const float4 v4 = *(const float4*)(src + db * 32 + i4 * 8 + h * 4);
        O[db][i4 * 4] = v4.x;
        O[db][i4 * 4 + 1] = v4.y;
        O[db][i4 * 4 + 2] = v4.z;
        O[db][i4 * 4 + 3] = v4.w;
      }
    const float* ml = A.mlst + ((size_t)bh * g.N + qrow) * 4;
    m_run = ml[0];
    l_run = ml[1 + h];
  }
  // s_waitcnt immediate (gfx9 encoding) waiting for lgkmcnt(0) only
  constexpr int kWaitLgkm0 = 0xC07F;
  // The Q operands and any resumed state were loaded into registers with
  // ordinary global loads.  Wait for them here, once: otherwise the
  // compiler's wait before their first use inside the loop would be a
  // vmcnt(0) on every iteration, which also waits for the next tile's loads.
  __builtin_amdgcn_s_waitcnt(0x3f70);

  const int ntile = (w.nkeys + KT - 1) / KT;
  // One step computes tile t (K in the K buffer, V in V buffer vb).  Barrier
  // A: every wave's copies of tile t have landed and every wave is done with
  // tile t-1, so V(t+1) is copied into the other V buffer; the scores read
  // the K buffer; barrier B: every wave is done with K(t), so K(t+1) is
  // copied into it while the softmax and PV of tile t run.  Plain s_barrier
  // (no fence): ordering is explicit, each wave waits for its own copies and
  // LDS accesses before a barrier.
  auto step = [&](int t, int vb) {
    const uint16_t* kt = tiles[0];
    const uint16_t* vt = tiles[1 + vb];
    // positions first: the range walk may read global memory, and the wait
    // the compiler puts before its use also covers the copies issued
    // earlier, which are awaited next anyway
    if (t + 2 < ntile) fill_pos(t + 2);
    __builtin_amdgcn_s_waitcnt(0x3f70);  // vmcnt(0): K(t) and V(t) have landed
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_s_barrier();
    if (t + 1 < ntile) issue(t + 1, Vp, vdst(1 - vb));
    f32x16 S;
    if (wave_active) {
#pragma unroll
      for (int i = 0; i < 16; ++i) S[i] = 0.f;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const int c8 = (2 * ks + h) ^ kv_swz<D>(n);
        const bf16x8 kf = __builtin_bit_cast(bf16x8, *(const uint4*)(kt + (n * CH + c8) * 8));
        S = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qreg[ks], S, 0, 0, 0);
      }
    }
    // every wave's K reads are done before K(t+1) overwrites the buffer
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_s_barrier();
    if (t + 1 < ntile) issue(t + 1, Kp, kdst);
    if (wave_active) {
      // register i holds key (i/4)*8 + h*4 + i%4 of the tile
      float mt = -INFINITY;
      if ((t + 1) * KT > w.nkeys) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = t * KT + (i >> 2) * 8 + h * 4 + (i & 3);
          if (key >= w.nkeys) S[i] = -INFINITY;
        }
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) mt = fmaxf(mt, S[i]);
      mt = pair_max(mt) * sl2;
      const bool need = mt > m_run + 8.f;
      if (__ballot(need)) {
        const float m_new = need ? mt : m_run;
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int i = 0; i < 16; ++i) O[db][i] *= alpha;
      }
      // probabilities rounded to bf16 for the PV product; the row sum is
      // taken over the same rounded values (two per dot2), so O and l share
      // one set of weights
      bf16x8 P[2];
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          P[c][e] = (__bf16)__builtin_amdgcn_exp2f(fmaf(S[c * 8 + e], sl2, -m_run));
      typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
      const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const bf16x2 pp = {P[c][e], P[c][e + 1]};
          l_run = __builtin_amdgcn_fdot2_f32_bf16(pp, one2, l_run, false);
        }
      // V^T fragments (transposing reads), after the scores are consumed so
      // that the two never hold registers together
      const int grp = lane >> 4, gl = lane & 15;
      bf16x8 vf[NDB][2];
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const int dv = db * 32 + 16 * (grp & 1) + 4 * (gl & 3);
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const int key0 = 16 * c + 4 * h + (gl >> 2);
          const int key1 = key0 + 8;
          const v4i16 lo = lds_read_tr16(vt + (key0 * CH + ((dv >> 3) ^ kv_swz<D>(key0))) * 8 + (dv & 7));
          const v4i16 hi = lds_read_tr16(vt + (key1 * CH + ((dv >> 3) ^ kv_swz<D>(key1))) * 8 + (dv & 7));
          vf[db][c] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        }
      }
      // O^T += V^T P^T over the two 16-key chunks
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int c = 0; c < 2; ++c)
          O[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[db][c], P[c], O[db], 0, 0, 0);
    }
  };
  if (ntile > 0) fill_pos(0);
  if (ntile > 1) fill_pos(1);
  __syncthreads();
  if (ntile > 0) {
    issue(0, Kp, kdst);
    issue(0, Vp, vdst(0));
  }
  for (int t = 0; t < ntile; t += 2) {
    step(t, 0);
    if (t + 1 < ntile) step(t + 1, 1);
  }
  // every copy has landed before the block can end
  __builtin_amdgcn_s_waitcnt(0x3f70);
  if (!qvalid) return;
  const float l_tot = pair_sum(l_run);
  if (MODE == MODE_PROBE) {
    float* dst = A.part + (((size_t)bh * g.M + w.tile * 64 + qr) * g.nsplit + w.split) * (D + 2);
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int dv = db * 32 + i4 * 8 + h * 4;
        *(float4*)(dst + dv) =
            make_float4(O[db][i4 * 4], O[db][i4 * 4 + 1], O[db][i4 * 4 + 2], O[db][i4 * 4 + 3]);
      }
    if (h == 0) {
      dst[D] = m_run;
      dst[D + 1] = l_tot;
    }
  } else {
    const float inv = 1.f / l_tot;
    if (MODE == MODE_SPARSE && !A.seg_last) {
      // hand the running state to the next key segment
      float* dst = A.osp + ((size_t)bh * g.N + qrow) * D;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          const int dv = db * 32 + i4 * 8 + h * 4;
          *(float4*)(dst + dv) =
              make_float4(O[db][i4 * 4], O[db][i4 * 4 + 1], O[db][i4 * 4 + 2], O[db][i4 * 4 + 3]);
        }
      float* ml = A.mlst + ((size_t)bh * g.N + qrow) * 4;
      if (h == 0) ml[0] = m_run;
      ml[1 + h] = l_run;
    } else if (MODE == MODE_SPARSE) {
      float* dst = A.osp + ((size_t)bh * g.N + qrow) * D;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          const int dv = db * 32 + i4 * 8 + h * 4;
          *(float4*)(dst + dv) = make_float4(O[db][i4 * 4] * inv, O[db][i4 * 4 + 1] * inv,
                                             O[db][i4 * 4 + 2] * inv, O[db][i4 * 4 + 3] * inv);
        }
    } else {
      uint16_t* dst = (uint16_t*)A.out + qbase + (int64_t)qrow * g.sn;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          const int dv = db * 32 + i4 * 8 + h * 4;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const __bf16 bv = (__bf16)(O[db][i4 * 4 + e] * inv);
            dst[dv + e] = __builtin_bit_cast(uint16_t, bv);
          }
        }
    }
  }
}

// Group-major copies of K and V (Sec. 4.3): position p of head bh holds row
// perm_kv[p].  Each row is moved as 16-byte pieces.
template <int D>
__global__ __launch_bounds__(256) void k_permute_kv(Geom g, const void* k, const void* v,
                                                    const int32_t* permk, uint16_t* kperm,
                                                    uint16_t* vperm) {
  constexpr int CH = D / 8, RPB = 256 / CH;
  const int bh = blockIdx.y, tid = threadIdx.x;
  const int p = blockIdx.x * RPB + tid / CH, c = tid % CH;
  if (p >= g.N) return;
  const int64_t base = kv_base(g, bh);
  const int src = permk[(size_t)bh * g.N + p];
  const uint4 kv = *(const uint4*)((const uint16_t*)k + base + (int64_t)src * g.sn + c * 8);
  const uint4 vv = *(const uint4*)((const uint16_t*)v + base + (int64_t)src * g.sn + c * 8);
  *(uint4*)(kperm + ((size_t)bh * g.N + p) * D + c * 8) = kv;
  *(uint4*)(vperm + ((size_t)bh * g.N + p) * D + c * 8) = vv;
}

// fp32 variant (VALU): one thread per query row, 32-key tiles staged in LDS.
template <int D, int MODE>
__global__ __launch_bounds__(64) void k_attn_f32(Geom g, AttnArgs A) {
  constexpr int KT = 32;
  __shared__ float Ks[KT][D + 1];
  __shared__ float Vs[KT][D + 1];
  __shared__ int srcrow[KT];
  const int bh = (MODE == MODE_PROBE) ? blockIdx.z : blockIdx.y;
  Work1 w;
  if (!get_work<MODE>(g, A, bh, w)) return;
  const int tid = threadIdx.x;
  const int64_t base = kv_base(g, bh), qbase = q_base(g, bh, g.gq);
  const float* Kp = (const float*)A.k + base;
  const float* Vp = (const float*)A.v + base;
  const float* Qp = (const float*)A.q + qbase;
  const bool qvalid = tid < w.nrows;
  const int qrow = qvalid ? row_of<MODE>(g, A, bh, w, tid) : 0;
  float qv[D], o[D];
#pragma unroll
  for (int c = 0; c < D; ++c) {
    qv[c] = qvalid ? Qp[(int64_t)qrow * g.sn + c] : 0.f;
    o[c] = 0.f;
  }
  const int2* rg = nullptr;
  int nr = 0;
  if (MODE == MODE_SPARSE) {
    rg = A.rng + ((size_t)bh * g.CQt + w.a) * g.CKt;
    nr = A.rng_cnt[(size_t)bh * g.CQt + w.a];
  }
  KeyCursor cur{0, 0};
  const float scale = 1.f / sqrtf((float)D);
  const float l2e = 1.4426950408889634f;
  float m_run = -INFINITY, l_run = 0.f;
  const int ntile = (w.nkeys + KT - 1) / KT;
  for (int t = 0; t < ntile; ++t) {
    if (tid < KT) {
      const int f = t * KT + tid;
      srcrow[tid] = (f < w.nkeys) ? key_row<MODE>(g, A, bh, w, f, cur, rg, nr) : -1;
    }
    __syncthreads();
    for (int i = tid; i < KT * D; i += 64) {
      const int r = i / D, c = i % D;
      const int src = srcrow[r];
      Ks[r][c] = src >= 0 ? Kp[(int64_t)src * g.sn + c] : 0.f;
      Vs[r][c] = src >= 0 ? Vp[(int64_t)src * g.sn + c] : 0.f;
    }
    __syncthreads();
    const int kn = min(KT, w.nkeys - t * KT);
    float s[KT];
    float mt = -INFINITY;
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      float acc = 0.f;
#pragma unroll
      for (int c = 0; c < D; ++c) acc = fmaf(qv[c], Ks[j][c], acc);
      s[j] = (j < kn) ? acc * scale * l2e : -INFINITY;
      mt = fmaxf(mt, s[j]);
    }
    const float m_new = fmaxf(m_run, mt);
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int c = 0; c < D; ++c) o[c] *= alpha;
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      const float p = exp2f(s[j] - m_new);
      l_run += p;
#pragma unroll
      for (int c = 0; c < D; ++c) o[c] = fmaf(p, Vs[j][c], o[c]);
    }
    __syncthreads();
  }
  if (!qvalid) return;
  if (MODE == MODE_PROBE) {
    float* dst = A.part + (((size_t)bh * g.M + w.tile * 64 + tid) * g.nsplit + w.split) * (D + 2);
    for (int c = 0; c < D; ++c) dst[c] = o[c];
    dst[D] = m_run;
    dst[D + 1] = l_run;
  } else if (MODE == MODE_SPARSE) {
    float* dst = A.osp + ((size_t)bh * g.N + qrow) * D;
    for (int c = 0; c < D; ++c) dst[c] = o[c] / l_run;
  } else {
    float* dst = (float*)A.out + qbase + (int64_t)qrow * g.sn;
    for (int c = 0; c < D; ++c) dst[c] = o[c] / l_run;
  }
}

// Merge the key splits of the probe rows: O = sum_s o_s 2^(m_s - m) / sum_s l_s 2^(m_s - m).
// Kernels from here on take every query head in one launch: block index
// bq = j * BH + bh is query head j of K/V head bh, whose attend outputs are
// entry bq of the [G][BH] arrays and whose plan is entry bh.
__global__ __launch_bounds__(128) void k_probe_merge(Geom g, const float* part,
                                                     const int32_t* nprobes, float* odp) {
  const int p = blockIdx.x, bq = blockIdx.y, bh = bq % g.BH, c = threadIdx.x;
  if (p >= nprobes[bh] || c >= g.dv) return;
  const int D = g.dv;
  const float* src = part + ((size_t)bq * g.M + p) * g.nsplit * (D + 2);
  // both sweeps keep the split order; unrolled so that their loads overlap
  float m = -INFINITY;
#pragma unroll 8
  for (int s = 0; s < g.nsplit; ++s) m = fmaxf(m, src[(size_t)s * (D + 2) + D]);
  float l = 0.f, o = 0.f;
#pragma unroll 8
  for (int s = 0; s < g.nsplit; ++s) {
    const float* e = src + (size_t)s * (D + 2);
    const float f = exp2f(e[D] - m);
    l += e[D + 1] * f;
    o += e[c] * f;
  }
  odp[((size_t)bq * g.M + p) * D + c] = o / l;
}

static AttnArgs make_args(const Work* w, const void* q, const void* k, const void* v, void* out) {
  AttnArgs a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  if (w) {
    a.osp = w->osp;
    a.part = w->part;
    a.chunks = w->chunks;
    a.nchunks = w->nchunks;
    a.permq = w->permq;
    a.offq = w->offq;
    a.permk = w->permk;
    a.rng = w->rng;
    a.rng_cnt = w->rng_cnt;
    a.probes = w->probes;
    a.nprobes = w->nprobes;
    a.kperm = w->kperm;
    a.vperm = w->vperm;
    a.mlst = w->mlst;
  }
  a.seg_lo = 0;
  a.seg_hi = 0x7fffffff;
  a.seg_first = 1;
  a.seg_last = 1;
  return a;
}

template <int D>
static void attend_d(const Geom& g, const Work* wq, const void* q, const void* k, const void* v,
                     void* out, hipStream_t s, hipEvent_t* ev) {
  const dim3 gp((g.M + 63) / 64, g.nsplit, g.BH);
  // query head j of every K/V head: its own Geom (Q and output rows) and
  // workspace view (attend outputs); the plan and the group-major K/V are shared
  auto gj = [&](int j) {
    Geom h = g;
    h.gq = j;
    return h;
  };
  if (g.bf16) {
    constexpr int CH = D / 8;
    k_permute_kv<D><<<dim3((g.N + 256 / CH - 1) / (256 / CH), g.BH), 256, 0, s>>>(
        g, k, v, wq[0].permk, wq[0].kperm, wq[0].vperm);
  }
  if (ev) (void)hipEventRecord(ev[0], s);
  for (int j = 0; j < g.G; ++j) {
    const AttnArgs a = make_args(&wq[j], q, k, v, out);
    if (g.bf16) {
      // one launch per key segment, so that all blocks in flight read the same
      // slice of K/V and it stays in L2
      for (int sg = 0; sg < g.nseg; ++sg) {
        AttnArgs as = a;
        as.seg_lo = (int)((int64_t)g.N * sg / g.nseg);
        as.seg_hi = (int)((int64_t)g.N * (sg + 1) / g.nseg);
        as.seg_first = sg == 0;
        as.seg_last = sg == g.nseg - 1;
        as.heads_per_xcd = g.BH % 8 == 0;
        const dim3 grid = as.heads_per_xcd ? dim3(8 * g.nchunk_max, g.BH / 8)
                                           : dim3(8 * g.nchunk_per_xcd, g.BH);
        k_attn_mfma<D, MODE_SPARSE><<<grid, 128, 0, s>>>(gj(j), as);
      }
    } else {
      k_attn_f32<D, MODE_SPARSE><<<dim3(g.nchunk_max, g.BH), 64, 0, s>>>(gj(j), a);
    }
  }
  if (ev) (void)hipEventRecord(ev[1], s);
  // the kernels below take all G * BH query heads in one launch (view of
  // query head 0, whose [G][BH] arrays continue with the other query heads)
  const int BQ = g.BH * g.G;
  if (g.M > 0) {
    for (int j = 0; j < g.G; ++j) {
      const AttnArgs a = make_args(&wq[j], q, k, v, out);
      if (g.bf16)
        k_attn_mfma<D, MODE_PROBE><<<gp, 128, 0, s>>>(gj(j), a);
      else
        k_attn_f32<D, MODE_PROBE><<<gp, 64, 0, s>>>(gj(j), a);
    }
    k_probe_merge<<<dim3(g.M, BQ), 128, 0, s>>>(g, wq[0].part, wq[0].nprobes, wq[0].odp);
  }
  if (ev) (void)hipEventRecord(ev[2], s);
  launch_fit_correct(g, wq[0], out, s, ev);
}

void launch_attend(const Geom& g, const Work* wq, const void* q, const void* k, const void* v,
                   void* out, hipStream_t s, hipEvent_t* ev) {
  if (g.d == 64)
    attend_d<64>(g, wq, q, k, v, out, s, ev);
  else
    attend_d<128>(g, wq, q, k, v, out, s, ev);
}

void launch_dense(const Geom& g, const void* q, const void* k, const void* v, void* out,
                  float* part, hipStream_t s) {
  (void)part;
  const AttnArgs a = make_args(nullptr, q, k, v, out);
  const dim3 gd((g.N + 63) / 64, g.BH);
  for (int j = 0; j < g.G; ++j) {  // every query head of each K/V head
    Geom h = g;
    h.gq = j;
    if (g.d == 64) {
      if (g.bf16)
        k_attn_mfma<64, MODE_DENSE><<<gd, 128, 0, s>>>(h, a);
      else
        k_attn_f32<64, MODE_DENSE><<<gd, 64, 0, s>>>(h, a);
    } else {
      if (g.bf16)
        k_attn_mfma<128, MODE_DENSE><<<gd, 128, 0, s>>>(h, a);
      else
        k_attn_f32<128, MODE_DENSE><<<gd, 64, 0, s>>>(h, a);
    }
  }
}

}  // namespace sparsepr
