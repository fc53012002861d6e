// Device-side sequence state: row layout of an ingest, KV append, lengths.
//
// The committed length of every slot and the tokens committed by the last
// verification live on the device, so a steady-state draft -> verify -> draft
// loop needs no host synchronisation: k_setup turns them into the packed row
// list (sequence, absolute position, token, tap row) of the next ingest.
#include "common.h"
#include "internal.h"

#include <algorithm>

namespace osp {

constexpr int kSetupThreads = kMaxBatch;

__global__ void __launch_bounds__(kSetupThreads) k_setup(SetupArgs a) {
  __shared__ int s_tot[4];
  const int b = threadIdx.x;
  const int lane = b & 63, wave = b >> 6;
  const bool act = b < a.B;
  int slot = 0, len = 0, n = 0;
  if (act) {
    slot = a.slots[b];
    len = a.slot_len[slot];
    n = a.explicit_rows ? a.n_new[b] : a.pend_n[slot];
    if (n < 1 || n > a.max_new) {
      atomicOr(a.err, 1u << 0);
      n = min(max(n, 1), a.max_new);
    }
  }
  // block drafting: the block's mask rows follow the sequence's new rows
  const int m = act ? a.extra : 0;
  // exclusive prefixes over the batch (integer scans: wave scan + wave totals) of the
  // rows (n + m) and of the new rows alone (packed tap rows)
  const int inc = wave_incl_scan<int>(n + m), incn = wave_incl_scan<int>(n);
  __shared__ int s_totn[4];
  if (lane == 63) { s_tot[wave] = inc; s_totn[wave] = incn; }
  __syncthreads();
  int before = 0, total = 0, beforen = 0;
  for (int w = 0; w < kSetupThreads / 64; ++w) {
    if (w < wave) { before += s_tot[w]; beforen += s_totn[w]; }
    total += s_tot[w];
  }
  const int cu = before + inc - (n + m);
  const int cun = beforen + incn - n;
  if (act) {
    a.cu[b] = cu;
    a.last_row[b] = cu + n - 1;
    a.committed[b] = len + n;
    a.bslot[b] = slot;
    a.ar_pos[b] = len + n;
    for (int j = 0; j < n; ++j) {
      const int r = cu + j;
      int t = a.explicit_rows ? a.new_tokens[cun + j] : a.pend_tok[(long)slot * a.pend_ld + j];
      if (t < 0 || t >= a.V_T) {
        atomicOr(a.err, 1u << 1);
        t = min(max(t, 0), a.V_T - 1);
      }
      a.ing_seq[r] = b;
      a.ing_pos[r] = len + j;
      a.ing_tok[r] = t;
      a.ing_tap[r] = a.taps_stride > 0 ? b * a.taps_stride + j : cun + j;
    }
    // the block's mask rows: the anchor's tap row (its conditioning input, broadcast)
    const int anchor_tap = a.taps_stride > 0 ? b * a.taps_stride + n - 1 : cun + n - 1;
    for (int j = 0; j < m; ++j) {
      const int r = cu + n + j;
      a.ing_seq[r] = b;
      a.ing_pos[r] = len + n + j;
      a.ing_tok[r] = a.mask;
      a.ing_tap[r] = anchor_tap;
    }
    if (m > 0) {
      for (int k = 0; k <= m; ++k) {
        a.blk_gather[b * (m + 1) + k] = cu + n - 1 + k;
        a.blk_temp[b * (m + 1) + k] = a.temp[b];
      }
    }
    const int cap = a.slot_nblocks[slot] * a.kv_block;
    if (len + n + (a.K > 0 ? a.K - 1 : 0) > cap) atomicOr(a.err, 1u << 2);
    a.slot_len[slot] = len + n;
    a.pend_n[slot] = 0;
  }
  if (b == 0) {
    a.cu[a.B] = total;
    a.n_rows[0] = total;
  }
  // ---- attention work list: every split but the last of each sequence covers
  //      split_len positions; those come first (sequence-major), then the last
  //      splits by decreasing length, so the longest blocks start first.  An item
  //      carries the sequence's slot, so that a block finds its page table without
  //      one more dependent load ---------------------------------------------------------
  if (a.attn_items) {
    __shared__ int s_last[kSetupThreads];
    const int nmax = act ? len + n + (a.K > 0 ? a.K - 1 : 0) : 0;
    const int ns = act ? (nmax + a.split_len - 1) / a.split_len : 0;
    const int nfull = ns > 0 ? ns - 1 : 0;
    const int last = act ? nmax - nfull * a.split_len : -1;
    s_last[b] = last;
    const int finc = wave_incl_scan<int>(nfull);
    __syncthreads();
    if (lane == 63) s_tot[wave] = finc;
    __syncthreads();
    int fbefore = 0, ftotal = 0;
    for (int w = 0; w < kSetupThreads / 64; ++w) {
      if (w < wave) fbefore += s_tot[w];
      ftotal += s_tot[w];
    }
    if (act) {
      const int f0 = fbefore + finc - nfull;
      for (int sp = 0; sp < nfull; ++sp) a.attn_items[f0 + sp] = b | (slot << 8) | (sp << 16);
      int rank = 0;
      for (int o = 0; o < a.B; ++o) rank += (s_last[o] > last || (s_last[o] == last && o < b)) ? 1 : 0;
      a.attn_items[ftotal + rank] = b | (slot << 8) | (nfull << 16);
    }
    if (b == 0) a.attn_n_items[0] = ftotal + a.B;
  }
}

void launch_setup(const SetupArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_setup, dim3(1), dim3(kSetupThreads), 0, st, a);
}

// Append n positions of precomputed (post-RoPE) keys and values for every layer.
// k, v: [n_layers][n][nkv][hd].  Positions start at the slot's current length.
template <typename T>
__global__ void k_kv_append(T* kv, const T* k, const T* v, int n_layers, int n, int nkv, int hd,
                            int kv_block, const int32_t* block_table, int slot, int max_blocks,
                            const int32_t* slot_len) {
  const long total = (long)n_layers * n * nkv * hd;
  const long blk_elems = kv_block_elems(n_layers, nkv, kv_block, hd);
  const int len = slot_len[slot];
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < total;
       i += (long)gridDim.x * blockDim.x) {
    long t = i;
    const int e = t % hd; t /= hd;
    const int g = t % nkv; t /= nkv;
    const int p = t % n; t /= n;
    const int l = (int)t;
    const int pos = len + p;
    const int blk = pos / kv_block, within = pos - blk * kv_block;
    if (blk >= max_blocks) continue;
    const long phys = block_table[(long)slot * max_blocks + blk];
    T* base = kv + phys * blk_elems;
    base[(((long)l * 2 + 0) * nkv + g) * kv_block * hd + kv_k_at(within, e, hd)] = k[i];
    base[(((long)l * 2 + 1) * nkv + g) * kv_block * hd + kv_v_at(within, e, kv_block)] = v[i];
  }
}

__global__ void k_add_len(int32_t* slot_len, int slot, int n) { slot_len[slot] += n; }

void launch_kv_append(int kvdtype, void* kv, const void* k, const void* v, int n_layers, int n,
                      int nkv, int hd, int kv_block, const int32_t* block_table, int slot,
                      int max_blocks, const int32_t* slot_len, int32_t* slot_len_out,
                      hipStream_t st) {
  const long total = (long)n_layers * n * nkv * hd;
  const int grid = (int)std::min<long>((total + 255) / 256, 4096);
  if (total > 0) {
    if (kvdtype == 1)
      hipLaunchKernelGGL(k_kv_append<bf16_t>, dim3(grid), dim3(256), 0, st,
                         reinterpret_cast<bf16_t*>(kv), reinterpret_cast<const bf16_t*>(k),
                         reinterpret_cast<const bf16_t*>(v), n_layers, n, nkv, hd, kv_block,
                         block_table, slot, max_blocks, slot_len);
    else
      hipLaunchKernelGGL(k_kv_append<float>, dim3(grid), dim3(256), 0, st,
                         reinterpret_cast<float*>(kv), reinterpret_cast<const float*>(k),
                         reinterpret_cast<const float*>(v), n_layers, n, nkv, hd, kv_block,
                         block_table, slot, max_blocks, slot_len);
  }
  hipLaunchKernelGGL(k_add_len, dim3(1), dim3(1), 0, st, slot_len_out, slot, n);
}

// Shorten a slot to min(length, len) and drop its pending ingest.
__global__ void k_set_len(int32_t* slot_len, int32_t* pend_n, int slot, int len) {
  slot_len[slot] = min(slot_len[slot], len);
  pend_n[slot] = 0;
}

void launch_set_len(int32_t* slot_len, int32_t* pend_n, int slot, int len, hipStream_t st) {
  hipLaunchKernelGGL(k_set_len, dim3(1), dim3(1), 0, st, slot_len, pend_n, slot, len);
}

__global__ void k_fill_i32(int32_t* p, int32_t v, long n) {
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
    p[i] = v;
}

void launch_fill_i32(int32_t* p, int32_t v, long n, hipStream_t st) {
  if (n <= 0) return;
  const int grid = (int)std::min<long>((n + 255) / 256, 1024);
  hipLaunchKernelGGL(k_fill_i32, dim3(grid), dim3(256), 0, st, p, v, n);
}

}  // namespace osp
