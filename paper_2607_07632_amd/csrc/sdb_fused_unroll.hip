// Instances of the fused pass: the stage loop written out, blocks of kMaxBlock threads.

#include "sdb_fused.h"

namespace sdb {

const void* pick_fused_unrolled(int terminal) {
    SDB_FUSED_TERMINALS(4, 2, false, kMaxBlock, kUnrollStages)
    return nullptr;
}

}  // namespace sdb
