// Host-side checks of libkvc's C ABI under AddressSanitizer and UndefinedBehaviorSanitizer (host code only; no GPU is
// needed and no kernel is launched).  Every device address below is fake and is only compared, never dereferenced:
// each call fails a host-side argument check or is host-only bookkeeping.  Exit status 0 when every expectation holds.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#include "kvc.h"

static int failures = 0;
#define EXPECT(cond)                                                          \
  do {                                                                        \
    if (!(cond)) {                                                            \
      std::fprintf(stderr, "FAILED line %d: %s\n", __LINE__, #cond);          \
      ++failures;                                                             \
    }                                                                         \
  } while (0)

static void* fake(uintptr_t off) { return reinterpret_cast<void*>(0x7F0000001000ull + off); }

struct Fixture {
  std::vector<void*> k, v;
  kvc_cache cache{};
  std::vector<kvc_item> items;
  kvc_batch batch{};
  Fixture(int n = 1, int L = 2, int H = 2, int d = 128, int T = 100, int rank = 16) {
    for (int l = 0; l < L; ++l) {
      k.push_back(fake(0x100000u * l));
      v.push_back(fake(0x800000u + 0x100000u * l));
    }
    cache.dtype = KVC_BF16;
    cache.num_layers = L;
    cache.num_kv_heads = H;
    cache.head_dim = d;
    cache.block_size = 16;
    cache.num_blocks = 64;
    cache.block_stride = 16 * H * d;
    cache.token_stride = H * d;
    cache.head_stride = d;
    cache.k_layers = k.data();
    cache.v_layers = v.data();
    items.resize(n);
    for (int i = 0; i < n; ++i) {
      kvc_item& it = items[i];
      std::memset(&it, 0, sizeof(it));
      it.num_tokens = T;
      it.src_offset = 0;
      it.dst_offset = 512;
      it.state.num_layers = L;
      it.state.num_kv_heads = H;
      it.state.head_dim = d;
      it.state.num_tokens = T;
      it.state.rank = rank;
      it.state.coef_dtype = KVC_BF16;
      it.state.coef = fake(0x4000000);
      it.state.basis = static_cast<float*>(fake(0x8000000));
    }
    batch.num_items = n;
    batch.items = items.data();
    batch.item_scratch = fake(0xC000000);
  }
  kvc_status apply() { return kvc_apply(&cache, &batch, 0, cache.num_layers, nullptr); }
};

int main() {
  EXPECT(kvc_version() == KVC_VERSION);
  for (int s = 0; s <= KVC_ERR_TOO_LARGE; ++s) EXPECT(std::strlen(kvc_status_str(static_cast<kvc_status>(s))) > 0);
  EXPECT(kvc_state_bytes(32, 8, 128, 32768, 32, KVC_BF16) == (size_t)512 * (32768 * 32 * 2 + 32 * 128 * 4 + 32 * 4));
  EXPECT(kvc_item_scratch_bytes(3) == 3 * sizeof(kvc_item) && kvc_item_scratch_bytes(-1) == 0);
  EXPECT(kvc_dense_bytes(-1, 8, 128, 10, KVC_BF16) == 0);

  {  // argument checks of kvc_apply
    Fixture f;
    EXPECT(kvc_apply(nullptr, &f.batch, 0, 1, nullptr) == KVC_ERR_NULL_ARG);
    f.cache.head_dim = 96;
    EXPECT(f.apply() == KVC_ERR_UNSUPPORTED);
    Fixture g;
    g.items[0].state.rank = 129;
    EXPECT(g.apply() == KVC_ERR_SHAPE);
    Fixture h;
    h.items[0].dst_offset = 50;  // destination rows overlap the source rows
    EXPECT(h.apply() == KVC_ERR_ALIAS);
    Fixture m;
    m.batch.item_scratch = fake(8);
    EXPECT(m.apply() == KVC_ERR_ALIGN);
    Fixture e;
    EXPECT(kvc_apply(&e.cache, &e.batch, 1, 1, nullptr) == KVC_OK);  // empty layer range: nothing to launch
  }
  {  // cross-item overlap sweep over many items (contiguous rows): disjoint ranges pass the checks
    Fixture f(200, 1, 1, 128, 5);
    f.cache.num_blocks = 4096;
    for (int i = 0; i < 200; ++i) {
      f.items[i].src_offset = 10 * i;
      f.items[i].dst_offset = 4000 + 10 * i;
      f.items[i].state.rank = 0;
    }
    f.items[150].dst_offset = 10 * 73 + 2;  // lands inside item 73's source rows
    EXPECT(f.apply() == KVC_ERR_ALIAS);
  }
  {  // the per-layer and per-head workspace queries and their refusals
    Fixture f(1, 2, 8, 128, 300, 32);
    f.items[0].state.grouping = KVC_GROUP_LAYER;
    EXPECT(kvc_fit_workspace_bytes(&f.cache, &f.batch, 0, 2) > 0);
    f.items[0].state.rank = 120;
    EXPECT(kvc_fit_workspace_bytes(&f.cache, &f.batch, 0, 2) == 0);
    EXPECT(kvc_fit_state(&f.cache, &f.batch, 0, 2, KVC_FIT_DELTA, fake(0), 1ull << 40, nullptr) ==
           KVC_ERR_UNSUPPORTED);
  }
  {  // chain checks
    kvc_state a{}, b{}, o{};
    for (kvc_state* s : {&a, &b, &o}) {
      s->num_layers = 2;
      s->num_kv_heads = 2;
      s->head_dim = 128;
      s->num_tokens = 100;
      s->rank = 8;
      s->coef_dtype = KVC_BF16;
      s->coef = fake(0x100000);
      s->basis = static_cast<float*>(fake(0x200000));
    }
    o.rank = 17;  // more than r1 + r2
    EXPECT(kvc_chain(&a, &b, &o, 0, 2, fake(0), 1ull << 30, nullptr) == KVC_ERR_SHAPE);
    o.rank = 8;  // o aliases a's buffers
    EXPECT(kvc_chain(&a, &b, &o, 0, 2, fake(0), 1ull << 30, nullptr) == KVC_ERR_ALIAS);
  }
  {  // gate: workspace and allocation-free size limit
    Fixture f(1, 128, 64, 128, 4096);
    f.cache.num_blocks = 300;
    std::vector<kvc_state> st(16, f.items[0].state);
    for (auto& s : st) s.num_layers = 128, s.num_kv_heads = 64, s.num_tokens = 4096, s.rank = 16;
    kvc_anchors an{16, 4000, st.data(), static_cast<float*>(fake(0x300000))};
    EXPECT(kvc_gate_workspace_bytes(&f.cache, &an, 2048, 0, 128) == KVC_NOALLOC_SCRATCH_BYTES);
    EXPECT(kvc_gate_distances_noalloc(&f.cache, &f.batch, &an, 2049, 0, 128, static_cast<float*>(fake(0x200000)),
                                      nullptr) == KVC_ERR_TOO_LARGE);
    EXPECT(kvc_gate_distances(&f.cache, &f.batch, &an, 100, 0, 128, static_cast<float*>(fake(0x200000)), fake(0), 16,
                              nullptr) == KVC_ERR_WORKSPACE);
  }
  {  // Eq. 10-11 decision on the host
    const float d2[2] = {1.0f, 1.0f};
    float g[2], h = 0.0f;
    EXPECT(kvc_gate_decide(d2, 2, 0.5f, 1.0f, g, &h) == 0 && h > 0.999f);  // uniform weights: entropy 1
    const float d3[3] = {0.0f, 30.0f, 30.0f};
    EXPECT(kvc_gate_decide(d3, 3, 0.5f, 1.0f, nullptr, &h) == 1 && h < 0.01f);
    EXPECT(kvc_gate_decide(d3, 1, 0.5f, 1.0f, g, &h) == 0 && h == 1.0f);  // fewer than two anchors
  }
  {  // pool bookkeeping: fill, use, evict the least used of the five oldest, many times over
    kvc_pool* p = kvc_pool_create(7);
    EXPECT(p != nullptr && kvc_pool_create(0) == nullptr);
    int64_t ev = 0;
    for (int64_t id = 0; id < 7; ++id) EXPECT(kvc_pool_insert(p, id, 100 + (int)id, &ev) == id && ev == -1);
    const int32_t used[3] = {0, 2, 4};
    EXPECT(kvc_pool_record_use(p, used, 3) == KVC_OK);
    EXPECT(kvc_pool_insert(p, 100, 50, &ev) == 1 && ev == 1);  // slots 0..4 oldest; 1 and 3 unused, 1 older
    std::vector<int32_t> slots(7);
    EXPECT(kvc_pool_eligible(p, 103, slots.data()) == 4);
    for (int64_t id = 200; id < 2200; ++id) {
      const int32_t s = kvc_pool_insert(p, id, (int)(id % 97), &ev);
      EXPECT(s >= 0 && s < 7);
      const int32_t one[1] = {(int32_t)(id % 7)};
      EXPECT(kvc_pool_record_use(p, one, 1) == KVC_OK);
    }
    const int32_t bad[1] = {9};
    EXPECT(kvc_pool_record_use(p, bad, 1) == KVC_ERR_SHAPE);
    int64_t aid = 0, uses = 0;
    int32_t len = 0;
    EXPECT(kvc_pool_slot(p, 3, &aid, &len, &uses) == KVC_OK && aid >= 200);
    EXPECT(kvc_pool_slot(p, 7, &aid, &len, &uses) == KVC_ERR_SHAPE);
    kvc_pool_destroy(p);
  }
  if (failures) std::fprintf(stderr, "%d expectation(s) failed\n", failures);
  else std::printf("abi_sanitize: all host checks passed under ASan/UBSan\n");
  return failures ? 1 : 0;
}
