// Call counters of the host-only HIP stand-in (fake_hip.cpp).
#pragma once

struct FakeHipCounters {
  long host_malloc = 0, host_free = 0, device_malloc = 0, device_free = 0;
  long event_create = 0, event_destroy = 0, event_record = 0, event_sync = 0;
  long memcpy_async = 0;
  long stream_create = 0, stream_wait = 0;
  long launches = 0;

  long allocations() const { return host_malloc + host_free + device_malloc + device_free +
                                    event_create + event_destroy + stream_create; }
};

extern FakeHipCounters g_fake_hip;
