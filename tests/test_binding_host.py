"""Host-side behaviour of the Python binding that needs no GPU."""


def test_device_guard_switches_only_when_needed(monkeypatch):
    # the binding makes a tensor's device current around each library call
    import torch

    import paper_2505_22918_amd as rt

    calls = []
    state = {"cur": 0}
    monkeypatch.setattr(rt, "_current_device", lambda: state["cur"])

    def set_device(i):
        calls.append(i)
        state["cur"] = i

    monkeypatch.setattr(torch.cuda, "set_device", set_device)

    class T:
        def __init__(self, d):
            self.d = d

        def get_device(self):
            return self.d

    with rt._on(T(0)):
        assert state["cur"] == 0
    assert calls == []
    with rt._on(T(3)):
        assert state["cur"] == 3
    assert calls == [3, 0] and state["cur"] == 0
    try:
        with rt._on(T(2)):
            raise KeyError("inside")
    except KeyError:
        pass
    assert state["cur"] == 0 and calls[-2:] == [2, 0]
