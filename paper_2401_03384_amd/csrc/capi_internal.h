// Status/exception bridge used by every extern "C" entry point.
#pragma once

#include <exception>
#include <new>
#include <string>

#include "common.h"

namespace ce {

void set_last_error(const std::string& msg);

// Run f(); map ce::Error and other exceptions to a status and a message.
template <typename F>
ce_status guard(F&& f) {
    try {
        f();
        return CE_OK;
    } catch (const Error& e) {
        set_last_error(e.what());
        return e.status;
    } catch (const std::bad_alloc&) {
        set_last_error("host out of memory");
        return CE_ERR_ARG;
    } catch (const std::exception& e) {
        set_last_error(e.what());
        return CE_ERR_ARG;
    } catch (...) {
        set_last_error("unknown error");
        return CE_ERR_ARG;
    }
}

}  // namespace ce
