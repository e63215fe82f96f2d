/* lora_status_string called from C with any int code (well defined in C). */
#include "lora_linear.h"

const char* status_text(int code) { return lora_status_string((lora_status)code); }
