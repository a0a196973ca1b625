// Host-side argument checks of every entry point of include/tq.h, for a
// build of the library's host code under AddressSanitizer (the device code
// is not part of this build).  Every call below is rejected on the host
// before any HIP call: the pointers are fake, aligned addresses that are
// never dereferenced, so this program must run where no GPU is visible.
// Exit status 0 when every call returns the expected status.  With
// --overflow it first writes one byte past a host heap block, so that a run
// can show the sanitizer is active.
#include <cstdint>
#include <cstdio>
#include <cstring>

#include "tq.h"

namespace {

int failures = 0;

void expect(const char* what, int got, int want) {
  if (got != want) {
    std::printf("FAIL %s: got %d, want %d\n", what, got, want);
    ++failures;
  }
}

const uintptr_t kFake = 0x7F0000000000ull;   // 256-byte aligned, never dereferenced
template <class T>
T* fake(uintptr_t off = 0) {
  return reinterpret_cast<T*>(kFake + off);
}

tq_matrix mat() {
  tq_matrix m;
  std::memset(&m, 0, sizeof m);
  m.n_out = 64;
  m.n_in = 256;
  m.group = TQ_GROUP;
  m.codes0 = fake<const uint8_t>();
  m.scale0 = fake<const uint16_t>(0x100000);
  return m;
}

int gemv(const tq_matrix& m, uintptr_t x = kFake + 0x200000, uintptr_t y = kFake + 0x300000, int flags = 0) {
  return tq_gemv(&m, reinterpret_cast<const uint16_t*>(x), reinterpret_cast<void*>(y), flags, nullptr);
}

}  // namespace

int main(int argc, char** argv) {
  if (argc > 1 && std::strcmp(argv[1], "--overflow") == 0) {
    char* volatile p = new char[8];
    p[8] = 1;
    delete[] p;
  }
  expect("abi version", tq_abi_version(), 7);
  for (int s = 0; s < 6; ++s) expect("status string", tq_status_string((tq_status)s) != nullptr, 1);
  expect("unknown status string", std::strstr(tq_status_string((tq_status)42), "unknown") != nullptr, 1);

  // Matrix checks (through tq_gemv).
  {
    tq_matrix m = mat();
    m.group = 64;
    expect("group", gemv(m), TQ_ERR_UNSUPPORTED);
    m = mat(); m.reserved = 1; expect("reserved", gemv(m), TQ_ERR_SHAPE);
    m = mat(); m.n_out = 0; expect("n_out", gemv(m), TQ_ERR_SHAPE);
    m = mat(); m.n_in = 100; expect("n_in % 128", gemv(m), TQ_ERR_SHAPE);
    m = mat(); m.n_in = 0; expect("n_in 0", gemv(m), TQ_ERR_SHAPE);
    m = mat(); m.n_in = 128 * (TQ_MAX_GROUPS_PER_ROW + 1); expect("groups per row", gemv(m), TQ_ERR_UNSUPPORTED);
    m = mat(); m.codes0 = nullptr; expect("codes0 null", gemv(m), TQ_ERR_NULL);
    m = mat(); m.scale0 = nullptr; expect("scale0 null", gemv(m), TQ_ERR_NULL);
    m = mat(); m.codes0 = fake<const uint8_t>(4); expect("codes0 align", gemv(m), TQ_ERR_ALIGN);
    m = mat(); m.scale0 = fake<const uint16_t>(1); expect("scale0 align", gemv(m), TQ_ERR_ALIGN);
    m = mat(); m.nnz1 = -1; expect("nnz1 < 0", gemv(m), TQ_ERR_SHAPE);
    m = mat(); m.nnz1 = 64 * 2 + 1; expect("nnz1 > N G", gemv(m), TQ_ERR_SHAPE);
    m = mat(); m.nnz1 = 3; expect("plane-1 pointers", gemv(m), TQ_ERR_NULL);
    m = mat(); m.nnz1 = 3;
    m.rowptr1 = fake<const int32_t>(2); m.gidx1 = fake<const uint16_t>(); m.codes1 = fake<const uint8_t>();
    m.offset1 = fake<const uint16_t>(); m.scale1 = fake<const uint16_t>();
    expect("rowptr1 align", gemv(m), TQ_ERR_ALIGN);
    m.rowptr1 = fake<const int32_t>(); m.codes1 = fake<const uint8_t>(4);
    expect("codes1 align", gemv(m), TQ_ERR_ALIGN);
    m = mat();
    expect("x null", gemv(m, 0), TQ_ERR_NULL);
    expect("y null", gemv(m, kFake, 0), TQ_ERR_NULL);
    expect("x align", gemv(m, kFake + 8), TQ_ERR_ALIGN);
    expect("y align", gemv(m, kFake, kFake + 2), TQ_ERR_ALIGN);
    expect("flags", gemv(m, kFake, kFake, 7), TQ_ERR_UNSUPPORTED);
    expect("matrix null", tq_gemv(nullptr, fake<const uint16_t>(), fake<void>(), 0, nullptr), TQ_ERR_NULL);
  }

  // Codec.
  expect("pack group", tq_pack(fake<const int8_t>(), 4, 64, fake<uint8_t>(), nullptr, nullptr), TQ_ERR_UNSUPPORTED);
  expect("pack n < 0", tq_pack(fake<const int8_t>(), -1, 128, fake<uint8_t>(), nullptr, nullptr), TQ_ERR_SHAPE);
  expect("pack null", tq_pack(nullptr, 4, 128, fake<uint8_t>(), nullptr, nullptr), TQ_ERR_NULL);
  expect("pack align", tq_pack(fake<const int8_t>(), 4, 128, fake<uint8_t>(4), nullptr, nullptr), TQ_ERR_ALIGN);
  expect("pack empty", tq_pack(nullptr, 0, 128, nullptr, nullptr, nullptr), TQ_OK);
  expect("unpack align", tq_unpack(fake<const uint8_t>(2), 4, 128, fake<int8_t>(), nullptr, nullptr), TQ_ERR_ALIGN);
  expect("unpack null", tq_unpack(fake<const uint8_t>(), 4, 128, nullptr, nullptr, nullptr), TQ_ERR_NULL);
  expect("validate counter", tq_validate(fake<const uint8_t>(), 4, 128, nullptr, nullptr), TQ_ERR_NULL);
  expect("validate align", tq_validate(fake<const uint8_t>(), 4, 128, fake<int32_t>(2), nullptr), TQ_ERR_ALIGN);
  {
    tq_matrix m = mat();
    expect("unpack_fp16 align", tq_unpack_fp16(&m, fake<uint16_t>(8), nullptr), TQ_ERR_ALIGN);
    expect("unpack_fp16 null", tq_unpack_fp16(&m, nullptr, nullptr), TQ_ERR_NULL);
  }

  // Grouped GEMV and small batch.
  {
    tq_matrix ms[3] = {mat(), mat(), mat()};
    ms[1].n_in = 512;
    void* ys[3] = {fake<void>(), fake<void>(), fake<void>()};
    expect("grouped K differs", tq_gemv_grouped(ms, 3, fake<const uint16_t>(), ys, 0, nullptr), TQ_ERR_SHAPE);
    expect("grouped n 0", tq_gemv_grouped(ms, 0, fake<const uint16_t>(), ys, 0, nullptr), TQ_ERR_SHAPE);
    expect("grouped n 9", tq_gemv_grouped(ms, 9, fake<const uint16_t>(), ys, 0, nullptr), TQ_ERR_SHAPE);
    void* ys0[1] = {nullptr};
    expect("grouped y null", tq_gemv_grouped(ms, 1, fake<const uint16_t>(), ys0, 0, nullptr), TQ_ERR_NULL);
    tq_matrix m = mat();
    expect("batch 0", tq_gemm_smallbatch(&m, fake<const uint16_t>(), 0, fake<void>(), 0, nullptr), TQ_ERR_SHAPE);
    expect("batch 65", tq_gemm_smallbatch(&m, fake<const uint16_t>(), TQ_MAX_BATCH + 1, fake<void>(), 0, nullptr),
           TQ_ERR_SHAPE);
    expect("batch X align", tq_gemm_smallbatch(&m, fake<const uint16_t>(2), 4, fake<void>(), 0, nullptr), TQ_ERR_ALIGN);
  }

  // Ternarisation.
  {
    auto call = [](const uint16_t* w, int64_t n, int32_t group, const int32_t* rec, int64_t nnz, int32_t iters,
                   int8_t* t0, uint16_t* s0, int8_t* t1, uint16_t* mu, uint16_t* s1, uint16_t* m0, double* e) {
      return (int)tq_ternarize(w, n, group, rec, nnz, iters, t0, s0, t1, mu, s1, m0, e, nullptr);
    };
    const uint16_t* W = fake<const uint16_t>();
    int8_t* T0 = fake<int8_t>();
    uint16_t* S0 = fake<uint16_t>();
    expect("ternarize group", call(W, 4, 64, nullptr, 0, 2, T0, S0, nullptr, nullptr, nullptr, nullptr, nullptr),
           TQ_ERR_UNSUPPORTED);
    expect("ternarize n", call(W, -1, 128, nullptr, 0, 2, T0, S0, nullptr, nullptr, nullptr, nullptr, nullptr),
           TQ_ERR_SHAPE);
    expect("ternarize iters", call(W, 4, 128, nullptr, 0, 1025, T0, S0, nullptr, nullptr, nullptr, nullptr, nullptr),
           TQ_ERR_SHAPE);
    expect("ternarize empty", call(nullptr, 0, 128, nullptr, 0, 2, nullptr, nullptr, nullptr, nullptr, nullptr,
                                   nullptr, nullptr), TQ_OK);
    expect("ternarize w null", call(nullptr, 4, 128, nullptr, 0, 2, T0, S0, nullptr, nullptr, nullptr, nullptr,
                                    nullptr), TQ_ERR_NULL);
    expect("ternarize records", call(W, 4, 128, nullptr, 3, 2, T0, S0, nullptr, nullptr, nullptr, nullptr, nullptr),
           TQ_ERR_NULL);
    expect("ternarize w align", call(fake<const uint16_t>(8), 4, 128, nullptr, 0, 2, T0, S0, nullptr, nullptr,
                                     nullptr, nullptr, nullptr), TQ_ERR_ALIGN);
  }

  // Two-plane selection.
  {
    const int64_t ws = tq_select_workspace_bytes(64 * 32);
    expect("workspace bytes", ws > 0 && ws % 256 == 0, 1);
    expect("workspace bytes < 0", (int)tq_select_workspace_bytes(-1), 0);
    auto call = [&](int64_t n_out, int32_t G, int64_t nnz, size_t wb, const double* e) {
      return (int)tq_select_two_plane(e, n_out, G, nnz, fake<int32_t>(), fake<int32_t>(), fake<uint16_t>(),
                                      fake<void>(), wb, nullptr);
    };
    const double* E = fake<const double>();
    expect("select n_out", call(0, 32, 10, ws, E), TQ_ERR_SHAPE);
    expect("select G", call(64, 257, 10, ws, E), TQ_ERR_SHAPE);
    expect("select nnz", call(64, 32, 64 * 32 + 1, ws, E), TQ_ERR_SHAPE);
    expect("select workspace", call(64, 32, 10, ws - 1, E), TQ_ERR_SHAPE);
    expect("select energy null", call(64, 32, 10, ws, nullptr), TQ_ERR_NULL);
    expect("select energy align", call(64, 32, 10, ws, fake<const double>(4)), TQ_ERR_ALIGN);
    expect("select noalloc n_out", (int)tq_select_two_plane_noalloc(E, 0, 32, 10, fake<int32_t>(), fake<int32_t>(),
                                                                    fake<uint16_t>(), nullptr), TQ_ERR_SHAPE);
    expect("select noalloc limit",
           (int)tq_select_two_plane_noalloc(E, TQ_SELECT_NOALLOC_MAX_GROUPS / 32 + 1, 32, 10, fake<int32_t>(),
                                            fake<int32_t>(), fake<uint16_t>(), nullptr), TQ_ERR_UNSUPPORTED);
  }

  // Chain.
  {
    tq_matrix ms[2] = {mat(), mat()};
    ms[1].n_in = 512;
    void* ys[2] = {fake<void>(), fake<void>()};
    tq_stage st;
    std::memset(&st, 0, sizeof st);
    st.mats = ms;
    st.n = 1;
    st.x = fake<const uint16_t>(0x400000);
    st.ys = ys;
    tq_chain_info info;
    std::memset(&info, 0, sizeof info);
    expect("chain no stages", tq_chain_plan(&st, 0, &info, nullptr, 0), TQ_ERR_SHAPE);
    expect("chain stages null", tq_chain_plan(nullptr, 1, &info, nullptr, 0), TQ_ERR_NULL);
    expect("chain info null", tq_chain_plan(&st, 1, nullptr, nullptr, 0), TQ_ERR_NULL);
    st.n = 2;
    expect("chain K differs", tq_chain_plan(&st, 1, &info, nullptr, 0), TQ_ERR_SHAPE);
    st.n = 1;
    st.flags = 3;
    expect("chain flags", tq_chain_plan(&st, 1, &info, nullptr, 0), TQ_ERR_UNSUPPORTED);
    st.flags = 0;
    st.x = fake<const uint16_t>(8);
    expect("chain x align", tq_chain_plan(&st, 1, &info, nullptr, 0), TQ_ERR_ALIGN);
    info.n_stages = 1;
    info.n_workgroups = 4;
    info.plan_bytes = 100;
    info.sync_bytes = 512;
    expect("chain bad info", tq_gemv_chain(fake<const void>(), fake<void>(), &info, nullptr), TQ_ERR_SHAPE);
    expect("chain sync bad info", tq_chain_sync_init(fake<void>(), &info, nullptr), TQ_ERR_SHAPE);
    expect("chain sync info null", tq_chain_sync_init(fake<void>(), nullptr, nullptr), TQ_ERR_NULL);
  }

  std::printf("%s: %d failure(s)\n", failures ? "FAILED" : "ok", failures);
  return failures ? 1 : 0;
}
