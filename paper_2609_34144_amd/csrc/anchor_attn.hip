// Routed block-sparse anchor attention on gfx950 (Sec. 4.4; App. B.4).
//
// Flash-style single pass with bf16 MFMA (v_mfma_f32_32x32x16_bf16) and fp32
// online softmax.  One workgroup = 8 waves = 256 queries of one (anchor, head);
// each wave owns one block of 32 queries.  The key sequence of the (anchor, head)
// is the concatenation [current segment (n0 tokens) ; routed chunk idx[0] ; ... ],
// walked in tiles of 64 keys.
//
// Two waves per SIMD, ping-pong: wave w runs on SIMD w % 4, so every SIMD holds
// one wave of group A (waves 0-3) and one of group B (waves 4-7).  The groups
// alternate between an MFMA interval (S = K Q^T of tile j and O += P V of tile
// j-1) and a softmax interval, half a tile apart, with a workgroup barrier between
// intervals: while one wave of a SIMD keeps the matrix core busy, the other issues
// the softmax's VALU work.  (Within one wave, VALU work between its own MFMAs is
// only partly hidden; across the two waves of a SIMD it is.)
//
// Data movement: every K and V tile is copied global -> LDS by the buffer unit
// (buffer_load_dwordx4 ... lds), so no registers or VALU work stage it.  Each
// lane of a copy instruction picks its source row and 16-byte chunk, which lets
// the LDS image be XOR-swizzled against bank conflicts even though the copy
// writes 1 KB contiguously.  Two K and two V buffers rotate; group A copies the
// K tiles and group B the V tiles, each at the start of its softmax interval.
//
// Per wave and tile:
//   S^T = K Q^T   A = K rows from LDS (ds_read_b128), B = Q^T held in registers
//                 for the whole kernel.  The 32x32 accumulator puts one query per
//                 lane column, so the online-softmax row max / row sum need only
//                 the lane's own values and one exchange with lane ^ 32.
//   O^T += V^T P^T  B = P^T straight from the S^T accumulators (converted to
//                 bf16; the contraction index order is free, so no data moves),
//                 A = V^T read from the row-major V tile with the transposing
//                 LDS load ds_read_b64_tr_b16.
// Blocks are renumbered so that the Q-tiles of one (anchor, head) land on the
// same XCD and share its L2 for the routed K/V.
#include "cast_common.h"

namespace cast {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) char lds_char;

constexpr int kBK = 64;    // keys per tile
constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
constexpr int kBQ = kWaves * 32;   // queries per workgroup: one block of 32 per wave
// operand reads issued this many MFMA steps ahead of their use
constexpr int kLookahead = 3;
// s_waitcnt vmcnt(0) that leaves expcnt and lgkmcnt free
constexpr int kVmcntBase = 0x0F70;
constexpr int kMaxKeff = kAttnMaxKeff;   // routed chunk indices cached in LDS
// The running max used for the exponentials moves only when the tile max exceeds
// it by more than this (log2 units): probabilities stay <= 2^8, harmless in fp32
// sums and bf16 operands, and the O rescale is skipped for most tiles.
constexpr float kMaxSlack = 8.0f;
// the lane sum of a tile's 32 probabilities up to which the running max may stay
constexpr float kSumBound = 256.0f;   // 2^kMaxSlack

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
  int nt_all;                    // 64-key tiles of the whole key sequence
  // work units (anchor, head, Q tile): the first n_full run whole, the last
  // n_split run as `split` pieces over disjoint key-tile ranges, each writing a
  // normalised fp32 partial output and its log2-domain log-sum-exp, merged after
  int n_full, n_split, split;
  float* part_o;                 // [n_split * split][kBQ][dh]
  float* part_lse;               // [n_split * split][kBQ]
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

// Block b runs on XCD b % 8, the blocks of one XCD in order of b / 8.  Each XCD
// takes a contiguous range of whole units (so the Q tiles of one (anchor, head),
// which read the same keys, share its L2), then a contiguous range of the pieces,
// which it runs last, in the partial round at the end.  Piece p is piece
// p / n_split of split unit n_full + p % n_split.  piece = -1 for a whole unit.
__device__ __forceinline__ void block_work(int b, int nblocks, int n_full, int n_split,
                                           int& unit, int& piece) {
  const int x = b & 7, j = b >> 3;
  const int qf = n_full >> 3, rf = n_full & 7;
  const int fx = qf + (x < rf ? 1 : 0);           // whole units on XCD x
  if (j < fx) {
    unit = x * qf + min(x, rf) + j;
    piece = -1;
    return;
  }
  const int qn = nblocks >> 3, rn = nblocks & 7;
  const int p = (x * qn + min(x, rn)) - (x * qf + min(x, rf)) + (j - fx);
  piece = p / n_split;
  unit = n_full + (p - piece * n_split);
}

// v_max3_f32 (the compiler forms it only from some max chains)
__device__ __forceinline__ float max3f(float x, float y, float z) {
  return __builtin_fmaxf(__builtin_fmaxf(x, y), z);
}

// Two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// Eight probabilities -> one bf16x8 MFMA operand (round to nearest even).
// (v_dot2_f32_bf16 is not used for the row sums: it waits for the matrix core,
// so beside the other wave's MFMAs it would stall the softmax.)
__device__ __forceinline__ bf16x8 pack8(const float* p) {
  return __builtin_bit_cast(bf16x8, u32x4{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                                          pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])});
}

constexpr int kBufDword3 = 0x00020000;   // 32-bit data format, gfx9-family V#

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tensor_rsrc(const void* base, long long bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0,
                                           (int)(unsigned)(bytes < 0xffffffffll ? bytes : 0xffffffffll),
                                           kBufDword3);
}

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

// Copy modes (MODE): 2 (aligned) no current segment and chunks of a multiple of
// 64 rows, so no tile crosses a chunk and each copy is one wave-uniform base plus
// the lane's fixed offset; 1 (fast) no current segment and chunks of >= 64 rows,
// so a tile meets at most two chunks; 0 the general path (current segment, short
// chunks), one chunk-slot lookup per row.
template <int DH, int MODE>
__global__ __launch_bounds__(kThreads, 1) void anchor_attn_kernel(AttnArgs a) {
  constexpr bool FAST = MODE >= 1, ALIGNED = MODE == 2;
  constexpr int CPR = DH / 8;                // 16-byte chunks per row
  constexpr int ROWB = DH * 2;               // bytes per row
  constexpr int KSL = DH / 8;                // 1-KB copy slots per K (or V) tile
  constexpr int NKS = KSL / 4;               // K (and V) slots per copying wave
  constexpr int RSTEP = 2048 / DH;           // tile rows between a wave's slots
  constexpr int ND = DH / 32;                // 32-row blocks of O^T
  constexpr int NSTEP = 2 * (DH / 16);       // MFMA steps per phase (= 4 ND)
  // separate objects, so the compiler can tell the copy targets from the buffers
  // being read and does not wait for in-flight copies before unrelated LDS reads
  __shared__ __attribute__((aligned(1024))) uint16_t lds_k0[kBK * DH];
  __shared__ __attribute__((aligned(1024))) uint16_t lds_k1[kBK * DH];
  __shared__ __attribute__((aligned(1024))) uint16_t lds_v0[kBK * DH];
  __shared__ __attribute__((aligned(1024))) uint16_t lds_v1[kBK * DH];
  __shared__ int sidx[kMaxKeff + 1];

  int unit, piece;
  block_work(blockIdx.x, a.nblocks, a.n_full, a.n_split, unit, piece);
  const int pair = unit / a.n_qt, qt = unit - pair * a.n_qt;
  // key tiles [tb, tb + nt) of the sequence's nt_all
  int tb = 0, nt = a.nt_all;
  if (piece >= 0) {
    tb = piece * a.nt_all / a.split;
    nt = (piece + 1) * a.nt_all / a.split - tb;
  }
  const int i = pair / a.H, h = pair - (pair / a.H) * a.H;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2;                 // 0: group A, 1: group B
  const int l32 = lane & 31, hf = lane >> 5;
  // a wave whose 32 queries all lie past S (in the last Q tile) skips its MFMA and
  // softmax work but still takes part in the copies and barriers; the padded
  // MFMAs would only draw power from the waves doing real work
  const bool live = qt * kBQ + wave * 32 < a.S;
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

  // ---- Q^T operand in registers: the lane holds query qt*BQ + wave*32 + l32,
  //      d = 16t + 8hf .. +8
  const int qi = qt * kBQ + wave * 32 + l32;
  bf16x8 qreg[DH / 16];
  {
    // rows past S load the last query; their outputs are never stored
    const int qc = qi < a.S ? qi : a.S - 1;
    const uint16_t* qp = a.q + (((long long)i * a.S + qc) * a.H + h) * DH + 8 * hf;
#pragma unroll
    for (int t = 0; t < DH / 16; ++t) {
      qreg[t] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(qp + 16 * t));
    }
  }
  __syncthreads();   // sidx visible to every wave
  // the first 64 routed chunks also sit one per lane in a register: the copy
  // cursors read them with v_readlane instead of waiting for LDS reads, which
  // queue behind the other group's operand reads
  const int sreg = sidx[lane < a.k_eff ? lane : a.k_eff];
  auto chunk_at = [&](int slot) __attribute__((always_inline)) -> int {
    if (slot < 64) return __builtin_amdgcn_readlane(sreg, slot);
    return __builtin_amdgcn_readfirstlane(sidx[slot]);
  };

  const unsigned row_bytes = (unsigned)(a.H * DH * 2), head_bytes = (unsigned)(h * DH * 2);

  // ---- copy slots.  The four waves of a group share the copy of a tile: wave
  //      w (mod 4) takes slots k = w + 4r, r < KSL / 4.  Slot k fills LDS chunks
  //      ci = 64 k + lane of its tile: row ci / CPR = brow + r RSTEP with
  //      brow = w 512/DH + lane / CPR, physical chunk lane % CPR, which holds logical
  //      chunk (lane % CPR) ^ swz(row).  Both swizzles depend on the row only
  //      through row mod CPR (K) or row mod 4 (V), which r does not change.
  const int cw = wave & 3;
  const int brow = cw * (512 / DH) + lane / CPR;
  const unsigned kofs = (unsigned)(((lane % CPR) ^ kswz(brow, CPR)) * 16);
  const unsigned vofs = (unsigned)(((lane % CPR) ^ vswz(brow, CPR)) * 16);
  auto copy16 = [&](__amdgpu_buffer_rsrc_t rs, uint16_t* dst, int r, unsigned off, unsigned soff)
      __attribute__((always_inline)) {
    // recomputed at each use (the laundering stops the compiler from keeping the
    // LDS bases of all buffers live in scalar registers across the loop)
    int sb = (cw + 4 * r) * 1024;
    asm volatile("" : "+s"(sb));
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(reinterpret_cast<char*>(dst) + sb), 16,
                                             (int)off, (int)soff, 0, 0);
  };
  // Fast modes: a history-only tile with chunks of >= 64 rows meets at most two
  // routed slots, whose rows are contiguous, so row j sits at
  // (j < split ? base0 : base1) + j * row_bytes with wave-uniform base0, base1,
  // split.  Rows past the end read real rows (of the repeated last slot); their
  // logits are masked to -inf and add nothing.
  struct TileMap { unsigned base0, base1; int split; };
  // Copy cursors: the tile being copied sits at row `off` of routed slot `s`
  // (chunks c0 = sidx[s], c1 = sidx[s + 1]); advancing by one tile crosses at most
  // one chunk boundary, so no division.
  struct Cursor { int s, off, c0, c1; };
  auto cursor_at = [&](int tile) __attribute__((always_inline)) -> Cursor {
    Cursor c;
    const int u0 = tile * kBK;
    c.s = u0 / a.Bv;
    c.off = u0 - c.s * a.Bv;
    c.c0 = chunk_at(c.s);
    c.c1 = chunk_at(c.s + 1);
    return c;
  };
  auto advance = [&](Cursor& c) __attribute__((always_inline)) {
    c.off += kBK;
    if (c.off >= a.Bv) {
      c.off -= a.Bv;
      c.s += 1;
      c.c0 = c.c1;
      c.c1 = chunk_at(c.s + 1);
    }
  };
  auto cur_map = [&](const Cursor& c) __attribute__((always_inline)) -> TileMap {
    TileMap m;
    m.base0 = (unsigned)(c.c0 * a.Bv + c.off) * row_bytes + head_bytes;
    m.base1 = (unsigned)(c.c1 * a.Bv + c.off - a.Bv) * row_bytes + head_bytes;
    m.split = a.Bv - c.off;
    return m;
  };
  // this wave's copies of tile `tile` of K (IsV = 0) or V (IsV = 1) into `dst`
  auto copy_tile = [&](auto is_v, int tile, const TileMap& m, uint16_t* dst) __attribute__((always_inline)) {
    constexpr bool IsV = decltype(is_v)::value != 0;
    const unsigned cofs = IsV ? vofs : kofs;
    const __amdgpu_buffer_rsrc_t rh = tensor_rsrc(IsV ? a.v : a.k, a.hist_bytes);
    static_for<0, NKS>([&](auto rr) {
      constexpr int r = decltype(rr)::value;
      const int row = brow + r * RSTEP;
      if constexpr (FAST) {
        const unsigned lane_off = (unsigned)row * row_bytes + cofs;
        if constexpr (ALIGNED) copy16(rh, dst, r, lane_off, m.base0);
        else copy16(rh, dst, r, (row < m.split ? m.base0 : m.base1) + lane_off, 0u);
      } else {
        // per-row chunk slot by multiply-shift
        int srow = tile * kBK + row;
        srow = srow < a.L ? srow : a.L - 1;
        const int rr2 = max(srow - a.n0, 0);
        const int slot = (int)(((unsigned long long)(unsigned)rr2 * a.bv_magic) >> 40);
        const int t = rr2 - slot * a.Bv;
        const unsigned hoff = (unsigned)(sidx[slot] * a.Bv + t) * row_bytes + head_bytes + cofs;
        // two copies under complementary lane masks (not an if/else, which would be
        // merged into one copy with a per-lane descriptor)
        if (srow < a.n0)
          copy16(tensor_rsrc(IsV ? a.vc : a.kc, a.cur_bytes), dst, r,
                 (unsigned)srow * row_bytes + head_bytes + cofs, 0u);
        if (srow >= a.n0) copy16(rh, dst, r, hoff, 0u);
      }
    });
  };
  // Copies of the tiles of j+1, at the start of the softmax interval of tile j:
  // group A copies K[j+1] (interval 2j+1), group B copies V[j+1] (interval
  // 2j+2), each into the buffer of tile j-1, and each waits for its copies at
  // the end of that interval.  Issuing a tile's copies holds the issuing waves
  // for about 16 cycles per 1-KB copy (the buffer unit's rate); split between
  // the groups, neither softmax interval grows past the MFMA phase beside it.
  // Both groups walk tiles j+1 = 1, 2, ... with one cursor per wave.
  Cursor cur{};
  if constexpr (FAST) cur = cursor_at(tb + min(1, nt - 1));
  auto own_copies = [&](int j, uint16_t* kdst, uint16_t* vdst) __attribute__((always_inline)) {
    if (j + 1 < nt) {
      const TileMap m = FAST ? cur_map(cur) : TileMap{};
      if (grp == 0) copy_tile(IC<0>{}, tb + j + 1, m, kdst);
      else copy_tile(IC<1>{}, tb + j + 1, m, vdst);
    }
    if constexpr (FAST) {
      if (j + 2 < nt) advance(cur);
    }
  };

  // ---- LDS read addresses (bytes within a tile)
  // K: lane reads row kb*32 + l32, logical chunk 2t + hf, stored at chunk
  // (2t + hf) ^ (l32 % CPR); as bytes that is kbase ^ 32t (the row offset is a
  // multiple of the row length, so the XOR only touches the chunk bits)
  const unsigned kbase = (unsigned)(l32 * ROWB + ((hf ^ kswz(l32, CPR)) * 16));
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
    vbase = (unsigned)(vr * ROWB + ((c ^ vswz(vr, CPR)) * 16) + 8 * (la & 1));
  }
  auto read_k = [&](const uint16_t* kt, int t, int kb) __attribute__((always_inline)) -> bf16x8 {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(
        reinterpret_cast<const char*>(kt) + (kbase ^ (32u * t)) + kb * 32 * ROWB));
  };
  auto read_v = [&](const uint16_t* vt, int db, int kb, int s2) __attribute__((always_inline)) -> bf16x8 {
    const lds_char* p = (const lds_char*)(vt) + (vbase ^ (64u * db)) + (32 * kb + 16 * s2) * ROWB;
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 8 * ROWB));
    return __builtin_bit_cast(bf16x8, u32x4{__builtin_bit_cast(u32x2, lo).x, __builtin_bit_cast(u32x2, lo).y,
                                            __builtin_bit_cast(u32x2, hi).x, __builtin_bit_cast(u32x2, hi).y});
  };

  f32x16 acc_o[ND];   // O^T of the wave's 32 queries (column = lane's query)
#pragma unroll
  for (int db = 0; db < ND; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc_o[db][e] = 0.0f;
  f32x16 sn[2];       // S^T of the current tile: keys kb*32 + 8(e/4) + 4hf + e%4
  bf16x8 pp[2][2];    // P^T operands of the previous tile, by (kb, 16-key half s2)
  // (a finite floor, so that an all -inf tile leaves m_run, l_run unchanged)
  float m_run = -1e30f, l_run = 0.0f;

  // ---- MFMA phase: S^T = K[j] Q^T and O^T += V^T[j-1] P^T[j-1], one S and one
  //      PV MFMA per step, operands read kLookahead steps ahead.  Step u: S chain
  //      kb = u % 2, d-chunk t = u / 2; PV chain db = u % ND with keys
  //      (kb, s2) = (u / (2 ND), (u / ND) % 2).  Consecutive MFMAs of one chain are
  //      at least four apart.
  auto mfma_phase = [&](const uint16_t* kt, const uint16_t* vt) __attribute__((always_inline)) {
    bf16x8 opk[NSTEP], opv[NSTEP];
    auto rd = [&](auto uu) __attribute__((always_inline)) {
      constexpr int u = decltype(uu)::value;
      opk[u] = read_k(kt, u / 2, u % 2);
      opv[u] = read_v(vt, u % ND, u / (2 * ND), (u / ND) % 2);
    };
    static_for<0, (kLookahead < NSTEP ? kLookahead : NSTEP)>([&](auto u) { rd(u); });
    static_for<0, NSTEP>([&](auto uu) {
      constexpr int u = decltype(uu)::value;
      if constexpr (u + kLookahead < NSTEP) rd(IC<u + kLookahead>{});
      sn[u % 2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(opk[u], qreg[u / 2], u < 2 ? f32x16{} : sn[u % 2],
                                                          0, 0, 0);
      constexpr int db = u % ND, kb = u / (2 * ND), s2 = (u / ND) % 2;
      acc_o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(opv[u], pp[kb][s2], acc_o[db], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  // ---- softmax phase of tile j: mask, exponentials against the running max,
  //      packed to the bf16 P^T operands and summed, running sum.  Every
  //      probability is at most the lane's sum of 32, so a sum <= 2^kMaxSlack
  //      (false for inf / NaN) shows that the running max may stay: no tile max
  //      is needed.  Otherwise (first tile, or a score more than kMaxSlack above
  //      the running max, or many close to it) the wave takes the exact path: row
  //      max (one exchange with the other half-wave), the running max moved only
  //      when the tile max exceeds it by more than kMaxSlack, exponentials again,
  //      and the O rescale.
  auto softmax_phase = [&](int j) __attribute__((always_inline)) {
    if (tb + j == a.nt_all - 1 && a.L != a.nt_all * kBK) {
      const int key0 = (tb + j) * kBK;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = key0 + kb * 32 + 8 * (e / 4) + 4 * hf + (e % 4);
          if (key >= a.L) sn[kb][e] = -INFINITY;
        }
    }
    // row sum in fp32 over four partial sums (short dependency chains), each
    // started from its first term (not 0 + p: the compiler keeps that add)
    float pe[32], rs4[4];
#pragma unroll
    for (int e = 0; e < 32; ++e) {
      pe[e] = __builtin_amdgcn_exp2f(fmaf(sn[e / 16][e % 16], a.sl2, -m_run));
      rs4[e % 4] = e < 4 ? pe[e] : rs4[e % 4] + pe[e];
    }
    float rs = (rs4[0] + rs4[1]) + (rs4[2] + rs4[3]);
    if (__ballot(!(rs <= kSumBound)) != 0ull) {
      float pm = max3f(sn[0][0], sn[0][1], sn[0][2]);
#pragma unroll
      for (int k = 1; k < 15; ++k) {
        const int v = 2 * k + 1;
        pm = max3f(pm, sn[v / 16][v % 16], sn[(v + 1) / 16][(v + 1) % 16]);
      }
      pm = fmaxf(pm, sn[1][15]);
      const u32x2 sw = __builtin_bit_cast(
          u32x2, __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, pm),
                                                  __builtin_bit_cast(unsigned, pm), false, false));
      const float mx = fmaxf(__builtin_bit_cast(float, sw.x), __builtin_bit_cast(float, sw.y));
      const float m_cand = fmaxf(m_run, mx * a.sl2);
      const bool up = m_cand > m_run + kMaxSlack;
      const float m_new = up ? m_cand : m_run;
      const float corr = __builtin_amdgcn_exp2f(m_run - m_new);
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        pe[e] = __builtin_amdgcn_exp2f(fmaf(sn[e / 16][e % 16], a.sl2, -m_new));
        rs4[e % 4] = e < 4 ? pe[e] : rs4[e % 4] + pe[e];
      }
      rs = (rs4[0] + rs4[1]) + (rs4[2] + rs4[3]);
      l_run *= corr;
      m_run = m_new;
      if (__ballot(up) != 0ull) {
#pragma unroll
        for (int db = 0; db < ND; ++db) acc_o[db] *= corr;
      }
    }
#pragma unroll
    for (int g = 0; g < 4; ++g) pp[g / 2][g % 2] = pack8(&pe[8 * g]);
    l_run += rs;
  };

  // ---- prologue: K[0]; tile -1 has P = 0 and a zeroed V buffer (P = 0 must not
  //      meet NaN in stale LDS)
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) pp[kb][s2] = bf16x8{};
  {
    u32x4* z = reinterpret_cast<u32x4*>(lds_v1);
    for (int x = tid; x < kBK * DH / 8; x += kThreads) z[x] = u32x4{0u, 0u, 0u, 0u};
  }
  {
    const TileMap m0 = FAST ? cur_map(cursor_at(tb)) : TileMap{};
    if (grp == 0) copy_tile(IC<0>{}, tb, m0, lds_k0);
    else copy_tile(IC<1>{}, tb, m0, lds_v0);
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // Group B runs one interval behind group A.  Interval 2j: A does the MFMAs of
  // tile j while B does the softmax of tile j-1; interval 2j+1: A the softmax of
  // tile j, B the MFMAs of tile j.  A copies K[j+1] at the start of interval
  // 2j+1, B copies V[j+1] at the start of interval 2j+2, each into a buffer that
  // no MFMA phase reads in that interval.
  if (grp == 1) __syncthreads();
  // One tile per call; K[j] in K buffer j%2, V[j-1] in V buffer (j-1)%2.  Every
  // call runs the same MFMA phase: at j = 0 it meets tile -1 (P = 0 and a zeroed V
  // buffer), at j = nt it computes a throw-away S from a stale K buffer.
  auto iter = [&](auto par, int j) __attribute__((always_inline)) {
    constexpr int P = decltype(par)::value;
    uint16_t* const kc = P == 0 ? lds_k0 : lds_k1;   // K[j]
    uint16_t* const kn = P == 0 ? lds_k1 : lds_k0;   // K[j-1]; then K[j+1]
    uint16_t* const vp = P == 0 ? lds_v1 : lds_v0;   // V[j-1]; then V[j+1]
    if (live) mfma_phase(kc, vp);
    __syncthreads();
    own_copies(j, kn, vp);
    if (j < nt && live) softmax_phase(j);
    // the copies of this interval land before the barrier publishes them: an
    // explicit wait, the same in both groups (the barrier's workgroup fence does
    // not reliably wait for copies into LDS)
    __builtin_amdgcn_s_waitcnt(kVmcntBase);
    __syncthreads();
  };
  int j = 0;
  for (; j + 1 <= nt; j += 2) {
    iter(IC<0>{}, j);
    iter(IC<1>{}, j + 1);
  }
  if (j <= nt) iter(IC<0>{}, j);
  if (grp == 0) __syncthreads();   // B's extra interval at the start

  // ---- epilogue: normalise, write O (bf16) and the log-sum-exp; a piece writes
  //      its normalised fp32 partial and log2-domain log-sum-exp instead
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = 1.0f / l_tot;
  if (piece >= 0) {
    if (qi < a.S) {
      const long long slot = (long long)(unit - a.n_full) * a.split + piece;
      const int ql = wave * 32 + l32;
      float* po = a.part_o + (slot * kBQ + ql) * DH + 4 * hf;
#pragma unroll
      for (int db = 0; db < ND; ++db)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4)
          *reinterpret_cast<f32x4*>(po + db * 32 + 8 * g4) =
              f32x4{acc_o[db][4 * g4 + 0] * inv, acc_o[db][4 * g4 + 1] * inv,
                    acc_o[db][4 * g4 + 2] * inv, acc_o[db][4 * g4 + 3] * inv};
      if (hf == 0) a.part_lse[slot * kBQ + ql] = m_run + __log2f(l_tot);
    }
  } else if (qi < a.S) {
    uint16_t* op = a.out + (((long long)i * a.S + qi) * a.H + h) * DH + 4 * hf;
#pragma unroll
    for (int db = 0; db < ND; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const u32x2 w = u32x2{pack_bf16x2(acc_o[db][4 * g4 + 0] * inv, acc_o[db][4 * g4 + 1] * inv),
                              pack_bf16x2(acc_o[db][4 * g4 + 2] * inv, acc_o[db][4 * g4 + 3] * inv)};
        *reinterpret_cast<u32x2*>(op + db * 32 + 8 * g4) = w;
      }
    if (a.lse && hf == 0)
      a.lse[((long long)i * a.H + h) * a.S + qi] = m_run * 0.69314718055994531f + logf(l_tot);
  }
}

// Merge of the pieces of each split unit: with l_p the log2-domain log-sum-exp
// and O_p the normalised output of piece p over its key range,
//   O = sum_p 2^(l_p - l_max) O_p / sum_p 2^(l_p - l_max),
//   log-sum-exp = ln 2 (l_max + log2 sum_p 2^(l_p - l_max)).
// One thread per (split unit, query of its tile, 4 channels).
template <int DH>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  constexpr int PER_Q = DH / 4, PER_UNIT = kBQ * PER_Q;
  const long long t = (long long)blockIdx.x * 256 + threadIdx.x;
  if (t >= (long long)a.n_split * PER_UNIT) return;
  const int u = (int)(t / PER_UNIT), rem = (int)(t - (long long)u * PER_UNIT);
  const int ql = rem / PER_Q, d4 = rem - ql * PER_Q;
  const int unit = a.n_full + u;
  const int pair = unit / a.n_qt, qt = unit - pair * a.n_qt;
  const int i = pair / a.H, h = pair - i * a.H;
  const int qi = qt * kBQ + ql;
  if (qi >= a.S) return;
  const long long slot0 = (long long)u * a.split;
  float lmax = -INFINITY;
  for (int p = 0; p < a.split; ++p) lmax = fmaxf(lmax, a.part_lse[(slot0 + p) * kBQ + ql]);
  float wsum = 0.0f;
  f32x4 acc{0.0f, 0.0f, 0.0f, 0.0f};
  for (int p = 0; p < a.split; ++p) {
    const float w = exp2f(a.part_lse[(slot0 + p) * kBQ + ql] - lmax);
    const f32x4 o = *reinterpret_cast<const f32x4*>(a.part_o + ((slot0 + p) * kBQ + ql) * DH + 4 * d4);
    wsum += w;
    acc += w * o;
  }
  const float inv = 1.0f / wsum;
  uint16_t* op = a.out + (((long long)i * a.S + qi) * a.H + h) * DH + 4 * d4;
  *reinterpret_cast<u32x2*>(op) = u32x2{pack_bf16x2(acc.x * inv, acc.y * inv), pack_bf16x2(acc.z * inv, acc.w * inv)};
  if (a.lse && d4 == 0)
    a.lse[((long long)i * a.H + h) * a.S + qi] = (lmax + log2f(wsum)) * 0.69314718055994531f;
}

template <int DH>
cast_status_t launch_dh(AttnArgs a, hipStream_t stream) {
  a.nblocks = a.n_full + a.n_split * a.split;
  if (a.n0 == 0 && a.Bv % kBK == 0)
    hipLaunchKernelGGL((anchor_attn_kernel<DH, 2>), dim3(a.nblocks), dim3(kThreads), 0, stream, a);
  else if (a.n0 == 0 && a.Bv >= kBK)
    hipLaunchKernelGGL((anchor_attn_kernel<DH, 1>), dim3(a.nblocks), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((anchor_attn_kernel<DH, 0>), dim3(a.nblocks), dim3(kThreads), 0, stream, a);
  if (a.n_split > 0) {
    const long long threads = (long long)a.n_split * kBQ * (DH / 4);
    hipLaunchKernelGGL((attn_merge_kernel<DH>), dim3((unsigned)((threads + 255) / 256)), dim3(256), 0,
                       stream, a);
  }
  return check_launch("anchor_attn");
}

}  // namespace

AttnSplitPlan attn_split_plan(int n_a, int S, int H, int dh, long long L, int cus) {
  constexpr long long kMaxSplit = 8, kMinPieceTiles = 16;
  const long long units = (long long)n_a * H * ((S + kBQ - 1) / kBQ);
  AttnSplitPlan p{(int)units, 0, 1, 0};
  if (cus <= 0) return p;
  const long long rem = units % cus;
  if (rem == 0) return p;
  const long long nt_all = (L + kBK - 1) / kBK;
  long long s = cus / rem;
  s = s < kMaxSplit ? s : kMaxSplit;
  s = s < nt_all / kMinPieceTiles ? s : nt_all / kMinPieceTiles;
  if (s < 2) return p;
  p.n_full = (int)(units - rem);
  p.n_split = (int)rem;
  p.split = (int)s;
  p.bytes = align_up((size_t)rem * s * kBQ * dh * 4) + align_up((size_t)rem * s * kBQ * 4);
  return p;
}

int device_cu_count() {
  // a benign race: concurrent first calls store the same value
  static int cache[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    return 0;
  }
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
      (void)hipGetLastError();
      return 0;
    }
    cache[dev] = n;
  }
  return cache[dev];
}

cast_status_t launch_anchor_attn(const void* q, const void* k_hist, const void* v_hist,
                                 const int32_t* idx, int k_eff, const void* k_cur,
                                 const void* v_cur, int n0, int n_a, int S, int H, int dh, int M,
                                 int Bv, float scale, void* out, float* lse_out,
                                 const AttnSplitPlan& plan, void* workspace, hipStream_t stream) {
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
  a.n_qt = (S + kBQ - 1) / kBQ;
  a.nt_all = (a.L + kBK - 1) / kBK;
  a.n_full = plan.n_full;
  a.n_split = plan.n_split;
  a.split = plan.split;
  if (plan.n_split > 0) {
    a.part_o = static_cast<float*>(workspace);
    a.part_lse = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                          align_up((size_t)plan.n_split * plan.split * kBQ * dh * 4));
  }
  switch (dh) {
    case 32: return launch_dh<32>(a, stream);
    case 64: return launch_dh<64>(a, stream);
    case 128: return launch_dh<128>(a, stream);
    default: return fail(CAST_ERR_UNSUPPORTED, "attn: dh %d", dh);
  }
}

}  // namespace cast
