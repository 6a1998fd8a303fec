// Routed block-sparse anchor attention on gfx950 (Sec. 4.4; App. B.4).
//
// Flash-style single pass with bf16 MFMA (v_mfma_f32_32x32x16_bf16) and fp32
// online softmax.  One workgroup = 4 waves = 128 queries of one (anchor, head);
// each wave owns 32 queries.  The key sequence of the (anchor, head) is the
// concatenation [current segment (n0 tokens) ; routed chunk idx[0] ; ... ], walked
// in tiles of 64 keys; each tile's rows are gathered from their chunk by index
// into LDS (double-buffered, one barrier per tile).
//
// Layout choices (per wave, per 64-key tile):
//   S^T = K Q^T   A = K tile from LDS (row-major, padded rows), B = Q^T held in
//                 registers for the whole kernel.  The 32x32 accumulator puts one
//                 query per lane column, so the row max / row sum of the online
//                 softmax need only the lane's own values and one exchange with
//                 lane^32.
//   O^T += V^T P^T  B = P^T straight from the S^T accumulators (converted to
//                 bf16; the contraction index order is free, so no data moves),
//                 A = V^T from an LDS copy of the V tile stored as
//                 [key/4][d][key%4] so each lane reads its 4-key runs as 8 bytes.
// Blocks are renumbered so that the Q-tiles of one (anchor, head) land on the
// same XCD and share its L2 for the routed K/V.
#include "cast_common.h"

namespace cast {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int kBK = 64;    // keys per tile
constexpr int kThreads = 256;
constexpr int kMaxKeff = kAttnMaxKeff;   // routed chunk indices cached in LDS

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
};

// Block b runs on XCD b % 8; give each XCD a contiguous range of logical blocks.
__device__ __forceinline__ int xcd_remap(int b, int nb) {
  const int per = nb / 8, rem = nb % 8;
  const int xcd = b % 8, j = b / 8;
  return (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + j;
}

// Address of key/value row r of the (anchor, head) sequence [current ; routed chunks].
// Rows past the end are clamped to the last row (their logits are masked, so they
// contribute exactly zero); chunk indices come from the LDS copy `sidx`.
template <int DH>
__device__ __forceinline__ const uint16_t* row_ptr(const AttnArgs& a, const uint16_t* hist,
                                                   const uint16_t* cur, const int* sidx, int r,
                                                   int h) {
  r = r < a.L ? r : a.L - 1;
  const unsigned rr = (unsigned)max(r - a.n0, 0);
  const unsigned slot = (unsigned)(((unsigned long long)rr * a.bv_magic) >> 40);
  const unsigned t = rr - slot * (unsigned)a.Bv;
  const uint16_t* hp = hist + (((long long)sidx[slot] * a.Bv + t) * a.H + h) * DH;
  const uint16_t* cp = cur + ((long long)r * a.H + h) * DH;
  return r < a.n0 ? cp : hp;
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

constexpr int kBufDword3 = 0x00020000;   // 32-bit data format, gfx9-family V#

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tensor_rsrc(const void* base, long long bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0,
                                           (int)(unsigned)(bytes < 0xffffffffll ? bytes : 0xffffffffll),
                                           kBufDword3);
}

template <int DH>
struct Tile {
  static constexpr int KSTR = DH + 8;                // padded K row (bf16 elements)
  static constexpr int K_ELEMS = kBK * KSTR;
  static constexpr int VG_STR = DH * 4 + 8;          // one 4-key group: [DH][4] + 16 B pad
  static constexpr int V_ELEMS = (kBK / 4) * VG_STR;  // [kBK/4][DH][4] with padded groups
  static constexpr int CPR = DH / 8;                 // 16-byte chunks per row
  static constexpr int RPP = kThreads / CPR;         // rows per load pass
  static constexpr int KPASS = kBK / RPP;            // K load passes per tile
  static constexpr int VITEMS = (kBK / 4) * CPR;     // V items (4 rows x 16 bytes)
  static constexpr int VPASS = (VITEMS + kThreads - 1) / kThreads;
};

template <int DH, int QB>
__global__ __launch_bounds__(kThreads, (QB == 1 ? 2 : 1)) void anchor_attn_kernel(AttnArgs a) {
  using T = Tile<DH>;
  constexpr int BQ = 4 * 32 * QB;   // queries per workgroup: 4 waves x QB blocks of 32
  __shared__ __attribute__((aligned(16))) uint16_t lds_k[2][T::K_ELEMS];
  __shared__ __attribute__((aligned(16))) uint16_t lds_v[2][T::V_ELEMS];
  __shared__ int sidx[kMaxKeff + 1];

  const int logical = xcd_remap(blockIdx.x, a.nblocks);
  const int pair = logical / a.n_qt, qt = logical - pair * a.n_qt;
  const int i = pair / a.H, h = pair - (pair / a.H) * a.H;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
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
    for (int t = 0; t < DH / 16; ++t)
      qreg[qb][t] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(qp + 16 * t));
  }
  __syncthreads();   // sidx visible to every wave

  // ---- tile loaders (global -> registers -> LDS)
  // Row j of tile `tile` is sequence row r = 64*tile + j: current segment rows
  // r < n0, then routed chunk rows.  When chunks hold >= 64 rows a tile meets at
  // most two chunks; their slots and indices are wave-uniform, so a lane's row
  // offset costs a handful of 32-bit ops.  Rows past the end are clamped to the
  // last row (their logits are masked to -inf and add nothing).
  const __amdgpu_buffer_rsrc_t rk = tensor_rsrc(a.k, a.hist_bytes);
  const __amdgpu_buffer_rsrc_t rv = tensor_rsrc(a.v, a.hist_bytes);
  const unsigned row_bytes = (unsigned)(a.H * DH * 2), head_bytes = (unsigned)(h * DH * 2);
  // History-only tiles (tile * 64 >= n0): with chunks of >= 64 rows a tile meets at
  // most two consecutive routed slots s0, s0 + 1, and rows are contiguous inside a
  // chunk, so row j of the tile sits at (j < split ? base0 : base1) + j * row_bytes
  // with wave-uniform base0, base1, split.  Rows past the end are harmless: they
  // read real rows of a routed chunk (sidx is padded) and their logits are masked.
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
  // general fallback (chunks shorter than a tile): per-row slot by multiply-shift
  auto hist_off_general = [&](int tile, int j) __attribute__((always_inline)) -> unsigned {
    int r = tile * kBK + j;
    r = r < a.L ? r : a.L - 1;
    const int rr = r - a.n0;
    const int slot = (int)(((unsigned long long)(unsigned)rr * a.bv_magic) >> 40);
    const int t = rr - slot * a.Bv;
    return (unsigned)(sidx[slot] * a.Bv + t) * row_bytes + head_bytes;
  };
  u32x4 kbuf[T::KPASS];
  u32x4 vbuf[T::VPASS][4];
  // V items: 16 four-key groups x CPR 16-byte chunks; within a wave, lanes vary the
  // group fastest (g = lane & 3) so the transposed LDS stores hit distinct banks
  auto v_item = [&](int it, int& g, int& ch) __attribute__((always_inline)) {
    g = (it & 3) + 4 * (it / (4 * T::CPR));
    ch = (it >> 2) % T::CPR;
  };
  auto load_tile = [&](int tile) __attribute__((always_inline)) {
    if (tile * kBK >= a.n0 && a.Bv >= kBK) {
      // history-only tile, chunks of >= 64 rows: buffer loads, 3 ops per row address
      const TileMap m = tile_map(tile);
#pragma unroll
      for (int p = 0; p < T::KPASS; ++p) {
        const int j = p * T::RPP + tid / T::CPR;
        const unsigned off = (j < m.split ? m.base0 : m.base1) + (unsigned)j * row_bytes +
                             (tid % T::CPR) * 16;
        kbuf[p] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rk, (int)off, 0, 0));
      }
#pragma unroll
      for (int p = 0; p < T::VPASS; ++p) {
        int g, ch;
        v_item(min(tid + p * kThreads, T::VITEMS - 1), g, ch);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int j = 4 * g + kk;
          const unsigned off = (j < m.split ? m.base0 : m.base1) + (unsigned)j * row_bytes + ch * 16;
          vbuf[p][kk] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rv, (int)off, 0, 0));
        }
      }
    } else if (tile * kBK >= a.n0) {
      // history-only tile, short chunks
#pragma unroll
      for (int p = 0; p < T::KPASS; ++p) {
        const unsigned off = hist_off_general(tile, p * T::RPP + tid / T::CPR) + (tid % T::CPR) * 16;
        kbuf[p] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rk, (int)off, 0, 0));
      }
#pragma unroll
      for (int p = 0; p < T::VPASS; ++p) {
        int g, ch;
        v_item(min(tid + p * kThreads, T::VITEMS - 1), g, ch);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const unsigned off = hist_off_general(tile, 4 * g + kk) + ch * 16;
          vbuf[p][kk] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rv, (int)off, 0, 0));
        }
      }
    } else {
      // tiles that touch the always-attended current segment: general row addresses
#pragma unroll
      for (int p = 0; p < T::KPASS; ++p)
        kbuf[p] = *reinterpret_cast<const u32x4*>(
            row_ptr<DH>(a, a.k, a.kc, sidx, tile * kBK + p * T::RPP + tid / T::CPR, h) +
            (tid % T::CPR) * 8);
#pragma unroll
      for (int p = 0; p < T::VPASS; ++p) {
        int g, ch;
        v_item(min(tid + p * kThreads, T::VITEMS - 1), g, ch);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          vbuf[p][kk] = *reinterpret_cast<const u32x4*>(
              row_ptr<DH>(a, a.v, a.vc, sidx, tile * kBK + 4 * g + kk, h) + ch * 8);
      }
    }
  };
  auto store_tile = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int p = 0; p < T::KPASS; ++p) {
      const int row = p * T::RPP + tid / T::CPR;
      *reinterpret_cast<u32x4*>(&lds_k[buf][row * T::KSTR + (tid % T::CPR) * 8]) = kbuf[p];
    }
#pragma unroll
    for (int p = 0; p < T::VPASS; ++p) {
      const int it = tid + p * kThreads;
      if (it < T::VITEMS) {
        int g, ch;
        v_item(it, g, ch);
        const u32x4 v0 = vbuf[p][0], v1 = vbuf[p][1], v2 = vbuf[p][2], v3 = vbuf[p][3];
        u32x4* dst = reinterpret_cast<u32x4*>(&lds_v[buf][g * T::VG_STR + ch * 8 * 4]);
        // word w of a row holds d = 8ch + 2w (low half) and 8ch + 2w + 1 (high half);
        // the LDS copy wants, per d, the 4 keys 4g..4g+3 side by side
#define CAST_VT(w)                                                                   \
  dst[w] = u32x4{__builtin_amdgcn_perm(v1[w], v0[w], 0x05040100u),                   \
                 __builtin_amdgcn_perm(v3[w], v2[w], 0x05040100u),                   \
                 __builtin_amdgcn_perm(v1[w], v0[w], 0x07060302u),                   \
                 __builtin_amdgcn_perm(v3[w], v2[w], 0x07060302u)};
        CAST_VT(0) CAST_VT(1) CAST_VT(2) CAST_VT(3)
#undef CAST_VT
      }
    }
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
  for (int qb = 0; qb < QB; ++qb) { m_run[qb] = -INFINITY; l_run[qb] = 0.0f; }

  const int ntiles = (a.L + kBK - 1) / kBK;
  load_tile(0);
  store_tile(0);
  __syncthreads();

  for (int tile = 0; tile < ntiles; ++tile) {
    const int buf = tile & 1;
    if (tile + 1 < ntiles) load_tile(tile + 1);

    // ---- S^T = K Q^T for the 64 keys of this tile: each K operand read from LDS
    //      feeds all QB query blocks
    f32x16 acc_s[QB][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc_s[qb][kb][e] = 0.0f;
      const uint16_t* kr = &lds_k[buf][(kb * 32 + l32) * T::KSTR + 8 * hf];
#pragma unroll
      for (int t = 0; t < DH / 16; ++t) {
        bf16x8 ka = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(kr + 16 * t));
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          acc_s[qb][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qreg[qb][t], acc_s[qb][kb], 0, 0, 0);
      }
    }
    // mask keys past the end of the sequence (last tile only)
    const int key0 = tile * kBK;
    if (key0 + kBK > a.L) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int key = key0 + kb * 32 + 8 * (e / 4) + 4 * hf + (e % 4);
            if (key >= a.L) acc_s[qb][kb][e] = -INFINITY;
          }
    }
    // ---- online softmax (log2 domain), one query per lane column
    bf16x8 pb[QB][2][2];
    float corr[QB];
    bool grew = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) mx = fmaxf(mx, acc_s[qb][kb][e]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[qb], mx * a.sl2);
      grew |= m_new > m_run[qb];
      corr[qb] = __builtin_amdgcn_exp2f(m_run[qb] - m_new);
      float rs = 0.0f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        float p[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          p[e] = __builtin_amdgcn_exp2f(fmaf(acc_s[qb][kb][e], a.sl2, -m_new));
          rs += p[e];
        }
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          u32x4 w = u32x4{pack_bf16x2(p[8 * s + 0], p[8 * s + 1]), pack_bf16x2(p[8 * s + 2], p[8 * s + 3]),
                          pack_bf16x2(p[8 * s + 4], p[8 * s + 5]), pack_bf16x2(p[8 * s + 6], p[8 * s + 7])};
          pb[qb][kb][s] = __builtin_bit_cast(bf16x8, w);
        }
      }
      l_run[qb] = l_run[qb] * corr[qb] + rs;
      m_run[qb] = m_new;
    }
    // rescale O only when some lane's running max moved (wave-uniform branch)
    if (__ballot(grew) != 0ull) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int db = 0; db < DH / 32; ++db)
#pragma unroll
          for (int e = 0; e < 16; ++e) acc_o[qb][db][e] *= corr[qb];
    }

    // ---- O^T += V^T P^T: each V^T operand read from LDS feeds all QB query blocks
#pragma unroll
    for (int db = 0; db < DH / 32; ++db) {
      const int d = db * 32 + l32;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          const int g = 8 * kb + 4 * s + hf;      // keys 4g..4g+3, then 4(g+2)..+3
          const u32x2 lo = *reinterpret_cast<const u32x2*>(&lds_v[buf][g * T::VG_STR + d * 4]);
          const u32x2 hi = *reinterpret_cast<const u32x2*>(&lds_v[buf][(g + 2) * T::VG_STR + d * 4]);
          bf16x8 va = __builtin_bit_cast(bf16x8, u32x4{lo.x, lo.y, hi.x, hi.y});
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            acc_o[qb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[qb][kb][s], acc_o[qb][db], 0, 0, 0);
        }
    }

    if (tile + 1 < ntiles) store_tile(buf ^ 1);
    __syncthreads();
  }

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

template <int DH, int QB>
cast_status_t launch_dh(AttnArgs a, hipStream_t stream) {
  a.n_qt = (a.S + 4 * 32 * QB - 1) / (4 * 32 * QB);
  a.nblocks = a.n_a * a.H * a.n_qt;
  hipLaunchKernelGGL((anchor_attn_kernel<DH, QB>), dim3(a.nblocks), dim3(kThreads), 0, stream, a);
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
  switch (dh) {
    case 32: return launch_dh<32, 1>(a, stream);
    case 64: return launch_dh<64, 1>(a, stream);
    case 128: return launch_dh<128, 1>(a, stream);
    default: return fail(CAST_ERR_UNSUPPORTED, "attn: dh %d", dh);
  }
}

}  // namespace cast
