// Instances of the fused pass: the stage loop written out, blocks of kBigBlock threads.

#include "sdb_fused.h"

namespace sdb {

const void* pick_fused_unrolled_big(int terminal) {
    SDB_FUSED_TERMINALS(4, 2, false, kBigBlock, kUnrollStages)
    return nullptr;
}

}  // namespace sdb
