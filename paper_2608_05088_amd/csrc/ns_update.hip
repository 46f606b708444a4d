// The Newton-Schulz update phase X' = s B' X (see ns_gemm.hip), compiled from
// the same main loop with its own stage geometry: 32-k stages in a four-slot
// LDS ring, each stage's direct loads spread between the MFMAs of the stage
// two ahead of it.  The update contracts over K = m' only, and measured on the
// GPT-2 Large set this ring beats two 64-k slots by 2.4%; the Gram and
// polynomial phases, whose longer contractions gain from fewer barriers, keep
// the two-slot ring of 64-k stages.
#define MALT_NS_BK 32
#define MALT_NS_STAGES 4
#define MALT_NS_UPDATE_TU 1
#include "ns_gemm.hip"
