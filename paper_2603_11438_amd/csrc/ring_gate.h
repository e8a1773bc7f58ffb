// Cross-stream ordering of ring kernel launches on one device.
//
// A ring kernel's workgroups wait on each other through flags, so a ring
// grid makes progress only once all of its workgroups are resident.  A plan
// checks at creation that its own grid fits on the device, but two ring
// grids launched on different streams can be dispatched interleaved: each
// then holds part of the device with spinning waves while the rest of its
// grid waits for room the other one occupies, and both end in the watchdog.
// The gate rules that out by never letting two ring grids overlap on one
// device.  Launches on one stream are ordered by the stream itself, and an
// event recorded between two kernels costs device time (a marker packet
// the command processor handles between them: about 2-3 us per launch on
// MI355X), so a device pays nothing while all its ring launches use one
// stream.  The first ring launch on a second stream waits, once, for the
// whole device (the earlier launches carry no event), and switches the
// device to ordered mode: from then on every ring launch records an event
// after itself, and a launch on another stream than the last one first
// makes its stream wait for that event.  Launches being captured into a
// graph are not gated (the graph's own edges order them; a graph replayed
// beside ring launches on other streams must be ordered by its caller).
//
// The policy is written against a small API so that it can be exercised on
// the host alone with a fake one; the library instantiates it with HIP.
//   Api::Stream, Api::Event                       handle types
//   int Api::capturing(Stream, bool *yes)         0 on success
//   int Api::sync_device()                        wait for all work of the device
//   int Api::create(Event *)                      0 on success
//   int Api::wait(Stream, Event)                  stream waits for the event
//   int Api::record(Event, Stream)                0 on success
#pragma once

#include <mutex>

namespace ar {

template <class Api, int kMaxDevices = 64>
class RingGate {
public:
    using Stream = typename Api::Stream;
    using Event = typename Api::Event;

    // Holds the device's gate from before the launch until after it, so that
    // launches from several host threads are ordered one at a time.
    class Ticket {
    public:
        Ticket() = default;
        Ticket(const Ticket &) = delete;
        Ticket &operator=(const Ticket &) = delete;
        ~Ticket() { release(); }
        void release()
        {
            if (lock_.owns_lock()) lock_.unlock();
        }

    private:
        friend class RingGate;
        std::unique_lock<std::mutex> lock_;
        int dev_ = -1;
        Stream stream_{};
        bool gated_ = false;
    };

    // Before a ring launch on `stream` of device `dev`.  Returns 0, or the
    // API's nonzero code (the launch must then not happen).
    int before(int dev, Stream stream, Ticket &t)
    {
        if (dev < 0 || dev >= kMaxDevices) return -1;
        State &st = state_[dev];
        t.lock_ = std::unique_lock<std::mutex>(st.mu);
        t.dev_ = dev;
        t.stream_ = stream;
        bool cap = false;
        int rc = Api::capturing(stream, &cap);
        if (rc != 0) return rc;
        t.gated_ = !cap;
        if (!t.gated_) return 0;
        if (!st.have_last || st.last == stream) return 0;
        if (!st.ordered) {
            // A second stream: the launches so far carry no event.
            if (!st.have_event) {
                rc = Api::create(&st.event);
                if (rc != 0) return rc;
                st.have_event = true;
            }
            rc = Api::sync_device();
            if (rc != 0) return rc;
            st.ordered = true;
            return 0;
        }
        return Api::wait(stream, st.event);
    }

    // After the launch was enqueued on the ticket's stream.
    int after(Ticket &t)
    {
        int rc = 0;
        if (t.gated_) {
            State &st = state_[t.dev_];
            if (st.ordered) rc = Api::record(st.event, t.stream_);
            if (rc == 0) {
                st.last = t.stream_;
                st.have_last = true;
            }
            // On failure the launch is enqueued but no event marks its end;
            // the caller reports the error (the device is then unusable).
        }
        t.release();
        return rc;
    }

    // Whether the device has switched to ordered mode (tests).
    bool ordered(int dev)
    {
        if (dev < 0 || dev >= kMaxDevices) return false;
        std::lock_guard<std::mutex> g(state_[dev].mu);
        return state_[dev].ordered;
    }

    // The stream of the device's last gated ring launch (tests).
    bool last_stream(int dev, Stream *out)
    {
        if (dev < 0 || dev >= kMaxDevices) return false;
        std::lock_guard<std::mutex> g(state_[dev].mu);
        if (!state_[dev].have_last) return false;
        *out = state_[dev].last;
        return true;
    }

private:
    struct State {
        std::mutex mu;
        Event event{};
        bool have_event = false;
        bool ordered = false;    // a second stream has been seen: record after every launch
        Stream last{};
        bool have_last = false;
    };
    State state_[kMaxDevices];
};

}  // namespace ar
