// Host-to-device feed for host-resident experts.
#include "pipeline.h"

namespace mp {

struct Pipeline::Impl {
};

Pipeline::Pipeline() : impl_(new Impl) {}
Pipeline::~Pipeline() { delete impl_; }

int Pipeline::index(const BlockTable&, const void*, const ExpertPtrs&, int, float*, hipStream_t,
                    std::string* err)
{
    *err = "host-pinned experts are not supported yet";
    return MP_E_UNSUPPORTED;
}

int Pipeline::merge(const BlockTable&, const MergeArgs&, const void*, const ExpertPtrs&, int,
                    const uint32_t*, void*, unsigned long long*, hipStream_t, mp_io_stats*,
                    std::string* err)
{
    *err = "host-pinned experts are not supported yet";
    return MP_E_UNSUPPORTED;
}

}  // namespace mp
