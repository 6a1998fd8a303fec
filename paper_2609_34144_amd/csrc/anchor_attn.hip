// Routed block-sparse anchor attention on gfx950 (Sec. 4.4; App. B.4).
//
// Flash-style single pass with bf16 MFMA (v_mfma_f32_32x32x16_bf16) and fp32
// online softmax.  One workgroup = 4 waves = 256 queries of one (anchor, head);
// each wave owns two blocks of 32 queries.  The key sequence of the (anchor,
// head) is the concatenation [current segment (n0 tokens) ; routed chunk idx[0] ;
// ... ], walked in tiles of 64 keys.
//
// Data movement: every K and V tile is copied global -> LDS by the buffer unit
// (buffer_load_dwordx4 ... lds), so no registers or VALU work stage it.  Each
// lane of a copy instruction picks its source row and 16-byte chunk, which lets
// the LDS image be XOR-swizzled against bank conflicts even though the copy
// writes 1 KB contiguously.  Two K and two V buffers rotate; one barrier per tile.
//
// Per wave and tile, for each query block:
//   S^T = K Q^T   A = K rows from LDS (ds_read_b128), B = Q^T held in registers
//                 for the whole kernel.  The 32x32 accumulator puts one query per
//                 lane column, so the online-softmax row max / row sum need only
//                 the lane's own values and one exchange with lane ^ 32.
//   O^T += V^T P^T  B = P^T straight from the S^T accumulators (converted to
//                 bf16; the contraction index order is free, so no data moves),
//                 A = V^T read from the row-major V tile with the transposing
//                 LDS load ds_read_b64_tr_b16.
// Each operand read from LDS feeds the MFMAs of both query blocks: with one block
// per wave the LDS read port, not the matrix core, was the limit.
// Schedule (per tile j, two straight-line phases of 32 MFMAs each):
//   phase 1: S[j] for both blocks      || softmax of S[j-1], block 1 (VALU)
//   phase 2: O += P[j-1] V[j-1], both   || softmax of S[j], block 0
// so the VALU work of the softmax overlaps the matrix cores inside one wave.
// Blocks are renumbered so that the Q-tiles of one (anchor, head) land on the
// same XCD and share its L2 for the routed K/V.
#include "cast_common.h"

namespace cast {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) char lds_char;

constexpr int kBK = 64;    // keys per tile
constexpr int kThreads = 256;
constexpr int kBQ = 256;   // queries per workgroup: 4 waves x 2 blocks of 32
constexpr int kMaxKeff = kAttnMaxKeff;   // routed chunk indices cached in LDS
// The running max used for the exponentials moves only when the tile max exceeds
// it by more than this (log2 units): probabilities stay <= 2^8, harmless in fp32
// sums and bf16 operands, and the O rescale is skipped for most tiles.
constexpr float kMaxSlack = 8.0f;

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* idx;
  const uint16_t* kc;
  const uint16_t* vc;
  uint16_t* out;
  float* lse;
  int n_a, S, H, M, Bv, n0, k_eff, L, n_qt, nblocks;
  unsigned long long bv_magic;   // ceil(2^40 / Bv): row / Bv = (row * magic) >> 40
  float sl2;                     // scale * log2(e)
  long long hist_bytes;          // extent of the K/V history tensors
  long long cur_bytes;           // extent of the current-segment K/V tensors
};

template <int V>
struct IC {
  static constexpr int value = V;
};

template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(IC<B>{});
    static_for<B + 1, E>(f);
  }
}

// Block b runs on XCD b % 8; give each XCD a contiguous range of logical blocks.
__device__ __forceinline__ int xcd_remap(int b, int nb) {
  const int per = nb / 8, rem = nb % 8;
  const int xcd = b % 8, j = b / 8;
  return (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + j;
}

// v_max3_f32 (the compiler forms it only from some max chains)
__device__ __forceinline__ float max3f(float x, float y, float z) {
  return __builtin_fmaxf(__builtin_fmaxf(x, y), z);
}

// Row sums add the bf16 probabilities that enter P V, two per v_dot2 with (1, 1).
constexpr bf16x2 kOnes2 = {(__bf16)1.0f, (__bf16)1.0f};

// Two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// Eight probabilities -> one bf16x8 MFMA operand; their bf16 values are added to
// `rs`.  (The pairs are kept as separate scalars: taking them back out of a
// 4-word vector for v_dot2 miscompiles with this toolchain.)
__device__ __forceinline__ bf16x8 pack8_sum(const float* p, float& rs) {
  const uint32_t w0 = pack_bf16x2(p[0], p[1]), w1 = pack_bf16x2(p[2], p[3]);
  const uint32_t w2 = pack_bf16x2(p[4], p[5]), w3 = pack_bf16x2(p[6], p[7]);
  rs = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w0), kOnes2, rs, false);
  rs = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w1), kOnes2, rs, false);
  rs = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w2), kOnes2, rs, false);
  rs = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w3), kOnes2, rs, false);
  return __builtin_bit_cast(bf16x8, u32x4{w0, w1, w2, w3});
}

constexpr int kBufDword3 = 0x00020000;   // 32-bit data format, gfx9-family V#

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tensor_rsrc(const void* base, long long bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0,
                                           (int)(unsigned)(bytes < 0xffffffffll ? bytes : 0xffffffffll),
                                           kBufDword3);
}

template <int DH>
struct Geo {
  static constexpr int CPR = DH / 8;                     // 16-byte chunks per row
  static constexpr int ROWB = DH * 2;                    // bytes per row
  static constexpr int TILEB = kBK * ROWB;               // bytes per K or V tile
  static constexpr int DPT = TILEB / (kThreads * 16);    // copy instructions per thread per tile
};

// LDS swizzles (chunk c of tile row r is stored at chunk c ^ swz(r)):
//  K: a ds_read_b128 of one logical chunk by 32 consecutive rows; XOR by r mod CPR
//     spreads any 16 consecutive rows over 16 distinct 16-byte bank groups.
//  V: a transposing read takes 4 consecutive rows x 32 bytes per 16 lanes, the
//     two 16-lane halves of 32 lanes 32 bytes apart; XOR by {0, 10, 4, 14}[r mod 4]
//     gives the 8 row segments of 32 lanes 8 distinct 32-byte bank groups.
__device__ __forceinline__ constexpr int kswz(int r, int cpr) { return r & (cpr - 1); }
__device__ __forceinline__ constexpr int vswz(int r, int cpr) {
  return ((2 * (r & 3)) ^ (8 * (r & 1))) & (cpr - 1);
}

// MODE 1 (fast): no current segment and chunks of >= 64 rows, so every tile takes
// the uniform two-chunk mapping and its copies can be issued inside the MFMA
// block.  MODE 2 (aligned): also chunks of a multiple of 64 rows, so no tile
// crosses a chunk and each copy is one uniform base plus the lane's fixed offset.
// MODE 0: the general path (current segment, short chunks).
// Each wave owns QB = 2 blocks of 32 queries: every K / V operand read from LDS
// feeds two MFMAs, which halves the LDS read traffic per MFMA (with one block
// per wave the LDS port, not the matrix core, is the limit).  The O accumulators
// live in the AGPR file; one workgroup runs per CU.
template <int DH, int MODE>
__global__ __launch_bounds__(kThreads, 1) void anchor_attn_kernel(AttnArgs a) {
  constexpr bool FAST = MODE >= 1, ALIGNED = MODE == 2;
  constexpr int QB = 2;
  using G = Geo<DH>;
  constexpr int BQ = kBQ;
  // separate objects, so the compiler can tell the copy targets from the buffers
  // being read and does not wait for in-flight copies before unrelated LDS reads
  __shared__ __attribute__((aligned(1024))) uint16_t lds_k0[kBK * DH];
  __shared__ __attribute__((aligned(1024))) uint16_t lds_k1[kBK * DH];
  __shared__ __attribute__((aligned(1024))) uint16_t lds_v0[kBK * DH];
  __shared__ __attribute__((aligned(1024))) uint16_t lds_v1[kBK * DH];
  __shared__ int sidx[kMaxKeff + 1];

  const int logical = xcd_remap(blockIdx.x, a.nblocks);
  const int pair = logical / a.n_qt, qt = logical - pair * a.n_qt;
  const int i = pair / a.H, h = pair - (pair / a.H) * a.H;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hf = lane >> 5;
  // routed chunk indices of this (anchor, head), clamped into [0, M)
  // (entry k_eff repeats the last one, so a tile's "next slot" always names a real chunk)
  if (a.k_eff > 0) {
    const int32_t* idx_ih = a.idx + ((long long)i * a.H + h) * a.k_eff;
    for (int j = tid; j <= a.k_eff; j += kThreads) {
      const int c = idx_ih[j < a.k_eff ? j : a.k_eff - 1];
      sidx[j] = c < 0 ? 0 : (c >= a.M ? a.M - 1 : c);
    }
  } else if (tid < 2) {
    sidx[tid] = 0;
  }

  // ---- Q^T operands in registers: for query block qb the lane holds query
  //      qt*BQ + (wave*QB + qb)*32 + l32, d = 16t + 8hf .. +8
  bf16x8 qreg[QB][DH / 16];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int qi = qt * BQ + (wave * QB + qb) * 32 + l32;
    // rows past S load the last query; their outputs are never stored
    const int qc = qi < a.S ? qi : a.S - 1;
    const uint16_t* qp = a.q + (((long long)i * a.S + qc) * a.H + h) * DH + 8 * hf;
#pragma unroll
    for (int t = 0; t < DH / 16; ++t) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(qp + 16 * t);
      // parked in the AGPR file (the MFMAs read their B operand there), which
      // leaves the VGPRs to S, P and the softmax
      unsigned x0, x1, x2, x3;
      asm volatile("v_accvgpr_write_b32 %0, %1" : "=a"(x0) : "v"(v.x));
      asm volatile("v_accvgpr_write_b32 %0, %1" : "=a"(x1) : "v"(v.y));
      asm volatile("v_accvgpr_write_b32 %0, %1" : "=a"(x2) : "v"(v.z));
      asm volatile("v_accvgpr_write_b32 %0, %1" : "=a"(x3) : "v"(v.w));
      qreg[qb][t] = __builtin_bit_cast(bf16x8, u32x4{x0, x1, x2, x3});
    }
  }
  __syncthreads();   // sidx visible to every wave

  const unsigned row_bytes = (unsigned)(a.H * DH * 2), head_bytes = (unsigned)(h * DH * 2);

  // ---- copy slots: instruction n of this wave fills LDS chunk
  //      ci = (wave * DPT + n) * 64 + lane of a tile, i.e. row ci / CPR and
  //      physical chunk ci % CPR, which holds logical chunk (ci % CPR) ^ swz(row)
  auto slot_row = [&](int n) __attribute__((always_inline)) -> int {
    return ((wave * G::DPT + n) * 64 + lane) / G::CPR;
  };
  auto slot_off = [&](int n, bool is_v) __attribute__((always_inline)) -> unsigned {
    const int r = slot_row(n), pc = lane % G::CPR;
    return (unsigned)((pc ^ (is_v ? vswz(r, G::CPR) : kswz(r, G::CPR))) * 16);
  };
  auto copy16 = [&](__amdgpu_buffer_rsrc_t rs, uint16_t* dst, int n, unsigned off, unsigned soff)
      __attribute__((always_inline)) {
    // recomputed at each use (the laundering stops the compiler from keeping the
    // LDS bases of all buffers live in scalar registers across the loop)
    int wbase = wave * G::DPT * 1024;
    asm volatile("" : "+s"(wbase));
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rs, (lds_void*)(reinterpret_cast<char*>(dst) + wbase + n * 1024), 16, (int)off, (int)soff, 0, 0);
  };
  // Row j of tile `tile` is sequence row r = 64*tile + j: current segment rows
  // r < n0, then routed chunk rows.  History-only tiles with chunks of >= 64 rows
  // meet at most two routed slots s0, s0 + 1, whose rows are contiguous, so row j
  // sits at (j < split ? base0 : base1) + j * row_bytes with wave-uniform base0,
  // base1, split.  Rows past the end read real rows (clamped, or of the padded
  // slot); their logits are masked to -inf and add nothing.
  struct TileMap { unsigned base0, base1; int split; };
  auto tile_map = [&](int tile) __attribute__((always_inline)) -> TileMap {
    const int u0 = tile * kBK - a.n0;                     // first chunk-part row of the tile
    const int s0 = u0 / a.Bv, tb = s0 * a.Bv;
    const int c0 = __builtin_amdgcn_readfirstlane(sidx[s0]);
    const int c1 = __builtin_amdgcn_readfirstlane(sidx[s0 + 1]);
    TileMap m;
    m.base0 = (unsigned)(c0 * a.Bv + (u0 - tb)) * row_bytes + head_bytes;
    m.base1 = (unsigned)(c1 * a.Bv + (u0 - tb - a.Bv)) * row_bytes + head_bytes;
    m.split = tb + a.Bv - u0;
    return m;
  };
  auto copy_fast = [&](auto is_v, const TileMap& m, int n, uint16_t* dst) __attribute__((always_inline)) {
    constexpr bool IsV = decltype(is_v)::value != 0;
    const int r = slot_row(n);
    const unsigned lane_off = (unsigned)r * row_bytes + slot_off(n, IsV);
    if constexpr (ALIGNED) {
      copy16(tensor_rsrc(IsV ? a.v : a.k, a.hist_bytes), dst, n, lane_off, m.base0);
    } else {
      copy16(tensor_rsrc(IsV ? a.v : a.k, a.hist_bytes), dst, n,
             (r < m.split ? m.base0 : m.base1) + lane_off, 0u);
    }
  };
  // Copy tile `tile` of K (is_v = 0) or V (is_v = 1) into `dst`.
  auto load_tile = [&](auto is_v, int tile, uint16_t* dst) __attribute__((always_inline)) {
    constexpr bool IsV = decltype(is_v)::value != 0;
    if (FAST || (tile * kBK >= a.n0 && a.Bv >= kBK)) {
      const TileMap m = tile_map(tile);
#pragma unroll
      for (int n = 0; n < G::DPT; ++n) copy_fast(is_v, m, n, dst);
    } else {
      // tiles that touch the current segment, or chunks shorter than a tile:
      // per-row slot by multiply-shift
      const __amdgpu_buffer_rsrc_t rh = tensor_rsrc(IsV ? a.v : a.k, a.hist_bytes);
#pragma unroll
      for (int n = 0; n < G::DPT; ++n) {
        int r = tile * kBK + slot_row(n);
        r = r < a.L ? r : a.L - 1;
        const unsigned co = slot_off(n, IsV);
        const int rr = max(r - a.n0, 0);
        const int slot = (int)(((unsigned long long)(unsigned)rr * a.bv_magic) >> 40);
        const int t = rr - slot * a.Bv;
        const unsigned hoff = (unsigned)(sidx[slot] * a.Bv + t) * row_bytes + head_bytes + co;
        // two copies under complementary lane masks (not an if/else, which would be
        // merged into one copy with a per-lane descriptor)
        if (r < a.n0)
          copy16(tensor_rsrc(IsV ? a.vc : a.kc, a.cur_bytes), dst, n,
                 (unsigned)r * row_bytes + head_bytes + co, 0u);
        if (r >= a.n0) copy16(rh, dst, n, hoff, 0u);
      }
    }
  };

  // ---- LDS read addresses (bytes within a tile)
  // K: lane reads row kb*32 + l32, logical chunk 2t + hf, stored at chunk
  // (2t + hf) ^ (l32 % CPR); as bytes that is kbase ^ 32t (the row offset is a
  // multiple of the row length, so the XOR only touches the chunk bits)
  const unsigned kbase = (unsigned)(l32 * G::ROWB + ((hf ^ kswz(l32, G::CPR)) * 16));
  // V (transposing read): within each 16-lane group gq = lane / 16, lane a supplies
  // row 4*(gq/2) + a/4 (+ 32kb + 16s + 8run) and columns d = 32db + 16(gq%2) + 4(a%4)
  // .. +4; the read returns to lane a the 4 rows' values at d = 32db + 16(gq%2) + a,
  // i.e. to every lane the column d = 32db + l32 for 4 consecutive keys.
  // As bytes: vbase ^ 64db (the row swizzle of vr only touches the chunk bits).
  unsigned vbase;
  {
    const int gq = lane >> 4, la = lane & 15;
    const int vr = 4 * (gq >> 1) + (la >> 2);
    const int c = 2 * (gq & 1) + ((la & 3) >> 1);
    vbase = (unsigned)(vr * G::ROWB + ((c ^ vswz(vr, G::CPR)) * 16) + 8 * (la & 1));
  }
  // operand reads: K rows (block kb, d-chunk t) and V^T (d-block db, keys of (kb, s))
  auto read_k = [&](const uint16_t* kt, int t, int kb) __attribute__((always_inline)) -> bf16x8 {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
        reinterpret_cast<const char*>(kt) + (kbase ^ (32u * t)) + kb * 32 * G::ROWB));
  };
  auto read_v = [&](const uint16_t* vt, int db, int kb, int s2) __attribute__((always_inline)) -> bf16x8 {
    const lds_char* p = (const lds_char*)(vt) + (vbase ^ (64u * db)) + (32 * kb + 16 * s2) * G::ROWB;
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 8 * G::ROWB));
    return __builtin_bit_cast(bf16x8, u32x4{__builtin_bit_cast(u32x2, lo).x, __builtin_bit_cast(u32x2, lo).y,
                                            __builtin_bit_cast(u32x2, hi).x, __builtin_bit_cast(u32x2, hi).y});
  };

  f32x16 acc_o[QB][DH / 32];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int db = 0; db < DH / 32; ++db)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc_o[qb][db][e] = 0.0f;
  float m_run[QB], l_run[QB];
#pragma unroll
  // (a finite floor, so that an all -inf tile leaves m_run, l_run unchanged)
  for (int qb = 0; qb < QB; ++qb) { m_run[qb] = -1e30f; l_run[qb] = 0.0f; }

  // new running max of block qb from this tile's row max `mx` (one exchange with
  // the other half-wave); the max used for the exponentials moves only by more
  // than kMaxSlack.  Returns whether it moved.
  auto new_max = [&](float mx, int qb, float& m_new, float& corr) __attribute__((always_inline)) -> bool {
    const u32x2 sw = __builtin_bit_cast(
        u32x2, __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, mx),
                                                __builtin_bit_cast(unsigned, mx), false, false));
    mx = fmaxf(__builtin_bit_cast(float, sw.x), __builtin_bit_cast(float, sw.y));
    const float m_cand = fmaxf(m_run[qb], mx * a.sl2);
    const bool up = m_cand > m_run[qb] + kMaxSlack;
    m_new = up ? m_cand : m_run[qb];
    corr = __builtin_amdgcn_exp2f(m_run[qb] - m_new);
    return up;
  };

  using SBlk = f32x16[2];      // S^T of one 32-query block and 64 keys
  using PBlk = bf16x8[2][2];   // its P^T operands
  // keys past the end of the sequence get logit -inf (the last tile, and the
  // throw-away tile nt)
  auto mask_tile = [&](SBlk& ss, int tile) __attribute__((always_inline)) {
    const int key0 = tile * kBK;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = key0 + kb * 32 + 8 * (e / 4) + 4 * hf + (e % 4);
        if (key >= a.L) ss[kb][e] = -INFINITY;
      }
  };
  using SAcc = SBlk[QB];
  using PAcc = PBlk[QB];
  constexpr int ND = DH / 32, NR = 2 * (DH / 16);   // operand reads per phase (K: 2 per t, V: 4 per db)
  constexpr int NM = QB * NR;                       // MFMAs per phase

  // ---- one phase = NM MFMAs sharing NR operand reads (each read feeds the QB
  //      query blocks), interleaved slice by slice with the softmax of one
  //      32-query block and, optionally, the tile copies.  A scheduling barrier
  //      closes each slice, so the VALU work issues while the matrix core runs.
  //      Softmax slices: 0-3 running max (v_max3 chain), 4 exchange with the other
  //      half-wave and new max, 5.. the 32 exponentials (packed to bf16 and summed
  //      every 8).
  //   IsPV = 0: S^T[qb] = K Q^T[qb] from the K tile `src` into `sn`.
  //   IsPV = 1: O^T[qb] += V^T P^T[qb] from the V tile `src` with operands `pp`.
  auto phase = [&](auto is_pv, auto do_mm, auto do_sm, auto do_copy, const uint16_t* src, SAcc& sn,
                   const PAcc& pp, SBlk& ss, PBlk& ps, float& corr, bool& up, int qbs, uint16_t* kdst,
                   const TileMap& mk, uint16_t* vdst, const TileMap& mv) __attribute__((always_inline)) {
    constexpr bool IsPV = decltype(is_pv)::value != 0, MM = decltype(do_mm)::value != 0;
    constexpr bool SM = decltype(do_sm)::value != 0;
    constexpr bool COPY = decltype(do_copy)::value != 0;
    constexpr int NSL = (MM ? NM : 0) > 32 ? NM : 32;
    constexpr int kLA = 2;
    bf16x8 op[NR];
    float pm = 0.0f, m_new = 0.0f, rs = 0.0f;
    float pe[32];
    auto read = [&](auto rr) __attribute__((always_inline)) {
      constexpr int r = decltype(rr)::value;
      if constexpr (!IsPV) op[r] = read_k(src, r / 2, r % 2);
      else op[r] = read_v(src, r % ND, r / (2 * ND), (r / ND) % 2);
    };
    auto mma = [&](auto uu) __attribute__((always_inline)) {
      constexpr int u = decltype(uu)::value, r = u / QB, qb = u % QB;
      if constexpr (!IsPV) {
        constexpr int t = r / 2, kb = r % 2;
        sn[qb][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op[r], qreg[qb][t], t == 0 ? f32x16{} : sn[qb][kb],
                                                             0, 0, 0);
      } else {
        constexpr int kb = r / (2 * ND), s2 = (r / ND) % 2, db = r % ND;
        acc_o[qb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op[r], pp[qb][kb][s2], acc_o[qb][db], 0, 0, 0);
      }
    };
    // first exponential of slice c >= 5: the 32 spread evenly over slices 5 .. NSL-1
    auto e_first = [](int c) constexpr { return c <= 5 ? 0 : ((c - 5) * 32) / (NSL - 5); };
    auto smx = [&](auto cc_) __attribute__((always_inline)) {
      constexpr int c = decltype(cc_)::value;
      if constexpr (c < 4) {
        static_for<4 * c, 4 * c + 4>([&](auto kk) {
          constexpr int k = decltype(kk)::value;
          if constexpr (k == 0) {
            pm = max3f(ss[0][0], ss[0][1], ss[0][2]);
          } else if constexpr (k < 15) {
            constexpr int v = 2 * k + 1;
            pm = max3f(pm, ss[v / 16][v % 16], ss[(v + 1) / 16][(v + 1) % 16]);
          } else {
            pm = fmaxf(pm, ss[1][15]);
          }
        });
      } else if constexpr (c == 4) {
        up = new_max(pm, qbs, m_new, corr);
      } else {
        constexpr int e0 = e_first(c), e1 = e_first(c + 1);
        static_for<e0, e1>([&](auto ee) {
          constexpr int e = decltype(ee)::value;
          pe[e] = __builtin_amdgcn_exp2f(fmaf(ss[e / 16][e % 16], a.sl2, -m_new));
          if constexpr (e % 8 == 7) {
            constexpr int g = e / 8;
            ps[g / 2][g % 2] = pack8_sum(&pe[8 * g], rs);
            // pinned here: the values are read only later, and the compiler would
            // otherwise sink this work out of the block it overlaps
            asm volatile("" ::"v"(ps[g / 2][g % 2]));
          }
          if constexpr (e == 31) {
            l_run[qbs] = l_run[qbs] * corr + rs;
            m_run[qbs] = m_new;
            asm volatile("" ::"v"(l_run[qbs]), "v"(corr));
          }
        });
      }
    };
    if constexpr (MM) static_for<0, kLA>([&](auto r) { read(r); });
    static_for<0, NSL>([&](auto uu) {
      constexpr int u = decltype(uu)::value;
      if constexpr (COPY && u < G::DPT) copy_fast(IC<0>{}, mk, u, kdst);
      if constexpr (COPY && u >= G::DPT && u < 2 * G::DPT) copy_fast(IC<1>{}, mv, u - G::DPT, vdst);
      if constexpr (MM) {
        // the read for operand r + kLA is issued with the first MFMA of operand r
        if constexpr (u % QB == 0 && u / QB + kLA < NR) read(IC<u / QB + kLA>{});
        if constexpr (u < NM) mma(uu);
      }
      if constexpr (SM) smx(uu);
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  const int nt = (a.L + kBK - 1) / kBK;
  SAcc sA, sB;        // S^T of even / odd tiles
  PAcc pA, pB;        // P^T of even / odd tiles
  float c0A = 1.0f, c1A = 1.0f, c0B = 1.0f, c1B = 1.0f;   // O rescale factors, by block and tile parity
  bool u0A = false, u1A = false, u0B = false, u1B = false;
  // tile -1 (odd): logits -inf and probabilities 0, so the first iteration's
  // softmax of its block 1 and its P V add nothing
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
    for (int e = 0; e < 16; ++e) sB[1][kb][e] = -INFINITY;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) pB[qb][kb][s2] = bf16x8{};
  }

  // Iteration j = 0 .. nt (tiles: K[j] in K buffer j%2, V[j-1] in V buffer (j-1)%2):
  //   copies K[j+1] -> K buffer (j+1)%2 and V[j] -> V buffer j%2 (their last
  //   readers ran in iteration j-1; past the end the last tile is copied again
  //   into a buffer that is not read for real data);
  //   phase 1: S[j] = K[j] Q^T (both blocks)     || softmax of S[j-1], block 1
  //   O rescale (both blocks by tile j-1's factors)
  //   phase 2: O += P[j-1] V[j-1] (both blocks)    || softmax of S[j], block 0
  // Iteration 0 meets tile -1 (all -inf, P = 0, V buffer zeroed); iteration nt
  // computes a throw-away S from a stale K tile whose block-0 softmax is fully
  // masked.  Every iteration runs the same straight-line phases.
  // Copy cursors of the fast path: the tile being copied sits at row `off` of
  // routed slot `s` (chunks c0 = sidx[s], c1 = sidx[s + 1]); advancing by one tile
  // crosses at most one chunk boundary (chunks have >= 64 rows), so no division.
  struct Cursor { int s, off, c0, c1; };
  auto cursor_at = [&](int tile) __attribute__((always_inline)) -> Cursor {
    Cursor c;
    const int u0 = tile * kBK;
    c.s = u0 / a.Bv;
    c.off = u0 - c.s * a.Bv;
    c.c0 = __builtin_amdgcn_readfirstlane(sidx[c.s]);
    c.c1 = __builtin_amdgcn_readfirstlane(sidx[c.s + 1]);
    return c;
  };
  auto advance = [&](Cursor& c) __attribute__((always_inline)) {
    c.off += kBK;
    if (c.off >= a.Bv) {
      c.off -= a.Bv;
      c.s += 1;
      c.c0 = c.c1;
      c.c1 = __builtin_amdgcn_readfirstlane(sidx[c.s + 1]);
    }
  };
  auto cur_map = [&](const Cursor& c) __attribute__((always_inline)) -> TileMap {
    TileMap m;
    m.base0 = (unsigned)(c.c0 * a.Bv + c.off) * row_bytes + head_bytes;
    m.base1 = (unsigned)(c.c1 * a.Bv + c.off - a.Bv) * row_bytes + head_bytes;
    m.split = a.Bv - c.off;
    return m;
  };
  Cursor cur_k{}, cur_v{};
  if constexpr (FAST) {
    cur_k = cursor_at(min(1, nt - 1));
    cur_v = cursor_at(0);
  }

  auto step = [&](auto par, int j, SAcc& sc, SAcc& sp, PAcc& pc, PAcc& pp, float& c0c, bool& u0c,
                  float& c0p, bool& u0p, float& c1p, bool& u1p) __attribute__((always_inline)) {
    constexpr int B = decltype(par)::value;
    const uint16_t* const kcur = B == 0 ? lds_k0 : lds_k1;   // K[j]
    uint16_t* const knext = B == 0 ? lds_k1 : lds_k0;        // K[j+1]
    uint16_t* const vcur = B == 0 ? lds_v0 : lds_v1;         // V[j]
    const uint16_t* const vprev = B == 0 ? lds_v1 : lds_v0;  // V[j-1]
    const int tk = min(j + 1, nt - 1), tv = min(j, nt - 1);
    __builtin_amdgcn_s_waitcnt(0);   // this wave's copies of the previous iteration landed
    __syncthreads();                 // ... and everyone's; previous readers are done
    if constexpr (!FAST) {
      load_tile(IC<0>{}, tk, knext);
      load_tile(IC<1>{}, tv, vcur);
    }
    if (j == nt) mask_tile(sp[1], j - 1);
    TileMap mk{}, mv{};
    if constexpr (FAST) {
      mk = cur_map(cur_k);
      mv = cur_map(cur_v);
    }
    phase(IC<0>{}, IC<1>{}, IC<1>{}, IC<FAST ? 1 : 0>{}, kcur, sc, pp, sp[1], pp[1], c1p, u1p, 1,
          knext, mk, vcur, mv);
    if constexpr (FAST) {
      if (j + 2 < nt) advance(cur_k);
      if (j + 1 < nt) advance(cur_v);
    }
    // O rescale before O += P[j-1] V[j-1]: block 0 by tile j-1's factor (phase 2 of
    // the previous iteration), block 1 by the one just computed
    if (__ballot(u0p || u1p) != 0ull) {
      // one accumulator at a time (they live in AGPRs; this bounds the VGPR copies)
      static_for<0, QB * ND>([&](auto kk) {
        constexpr int qb = decltype(kk)::value / ND, db = decltype(kk)::value % ND;
        acc_o[qb][db] *= (qb == 0 ? c0p : c1p);
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    if (j >= nt - 1) mask_tile(sc[0], j);
    phase(IC<1>{}, IC<1>{}, IC<1>{}, IC<0>{}, vprev, sc, pp, sc[0], pc[0], c0c, u0c, 0, nullptr, mk,
          nullptr, mv);
  };

  // zero the V buffer that iteration 0 reads as V[-1] (P[-1] = 0 must not meet NaN)
  {
    u32x4* z = reinterpret_cast<u32x4*>(lds_v1);
    for (int x = tid; x < kBK * DH / 8; x += kThreads) z[x] = u32x4{0u, 0u, 0u, 0u};
  }
  load_tile(IC<0>{}, 0, lds_k0);
  int j = 0;
  for (; j + 1 <= nt; j += 2) {
    step(IC<0>{}, j, sA, sB, pA, pB, c0A, u0A, c0B, u0B, c1B, u1B);
    step(IC<1>{}, j + 1, sB, sA, pB, pA, c0B, u0B, c0A, u0A, c1A, u1A);
  }
  if (j <= nt) step(IC<0>{}, j, sA, sB, pA, pB, c0A, u0A, c0B, u0B, c1B, u1B);

  // ---- epilogue: normalise, write O (bf16) and the log-sum-exp
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int qi = qt * BQ + (wave * QB + qb) * 32 + l32;
    const float l_tot = l_run[qb] + __shfl_xor(l_run[qb], 32);
    const float inv = 1.0f / l_tot;
    if (qi < a.S) {
      uint16_t* op = a.out + (((long long)i * a.S + qi) * a.H + h) * DH + 4 * hf;
#pragma unroll
      for (int db = 0; db < DH / 32; ++db)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const u32x2 w = u32x2{pack_bf16x2(acc_o[qb][db][4 * g4 + 0] * inv, acc_o[qb][db][4 * g4 + 1] * inv),
                                pack_bf16x2(acc_o[qb][db][4 * g4 + 2] * inv, acc_o[qb][db][4 * g4 + 3] * inv)};
          *reinterpret_cast<u32x2*>(op + db * 32 + 8 * g4) = w;
        }
      if (a.lse && hf == 0)
        a.lse[((long long)i * a.H + h) * a.S + qi] = m_run[qb] * 0.69314718055994531f + logf(l_tot);
    }
  }
}

template <int DH>
cast_status_t launch_dh(AttnArgs a, hipStream_t stream) {
  a.n_qt = (a.S + kBQ - 1) / kBQ;
  a.nblocks = a.n_a * a.H * a.n_qt;
  if (a.n0 == 0 && a.Bv % kBK == 0)
    hipLaunchKernelGGL((anchor_attn_kernel<DH, 2>), dim3(a.nblocks), dim3(kThreads), 0, stream, a);
  else if (a.n0 == 0 && a.Bv >= kBK)
    hipLaunchKernelGGL((anchor_attn_kernel<DH, 1>), dim3(a.nblocks), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((anchor_attn_kernel<DH, 0>), dim3(a.nblocks), dim3(kThreads), 0, stream, a);
  return check_launch("anchor_attn");
}

}  // namespace

cast_status_t launch_anchor_attn(const void* q, const void* k_hist, const void* v_hist,
                                 const int32_t* idx, int k_eff, const void* k_cur,
                                 const void* v_cur, int n0, int n_a, int S, int H, int dh, int M,
                                 int Bv, float scale, void* out, float* lse_out,
                                 hipStream_t stream) {
  AttnArgs a{};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k_hist);
  a.v = static_cast<const uint16_t*>(v_hist);
  a.idx = k_eff > 0 ? idx : nullptr;
  // keep every base pointer valid even for an empty segment (never dereferenced then)
  a.kc = static_cast<const uint16_t*>(n0 > 0 ? k_cur : k_hist);
  a.vc = static_cast<const uint16_t*>(n0 > 0 ? v_cur : v_hist);
  if (k_eff == 0) { a.k = a.kc; a.v = a.vc; }
  a.out = static_cast<uint16_t*>(out);
  a.lse = lse_out;
  a.n_a = n_a;
  a.S = S;
  a.H = H;
  a.M = M;
  a.Bv = Bv;
  a.n0 = n0;
  a.k_eff = k_eff;
  a.L = n0 + k_eff * Bv;
  a.bv_magic = ((1ull << 40) + (unsigned long long)Bv - 1) / (unsigned long long)Bv;
  a.sl2 = scale * 1.4426950408889634f;
  a.hist_bytes = k_eff > 0 ? (long long)M * Bv * H * dh * 2 : 0;
  a.cur_bytes = n0 > 0 ? (long long)n0 * H * dh * 2 : 0;
  switch (dh) {
    case 32: return launch_dh<32>(a, stream);
    case 64: return launch_dh<64>(a, stream);
    case 128: return launch_dh<128>(a, stream);
    default: return fail(CAST_ERR_UNSUPPORTED, "attn: dh %d", dh);
  }
}

}  // namespace cast
