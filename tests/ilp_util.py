"""Reader for the store/recompute example files under tests/golden/."""
EVENT_KINDS = ("alloc", "free", "produce", "drop", "recompute", "recompute_done", "release", "path")


def read_ilp_case(path):
    arrays, events, limit, expect = [], [], None, None
    with open(path) as f:
        for line in f:
            line = line.split("#", 1)[0].split()
            if not line:
                continue
            key = line[0]
            if key == "array":
                arrays.append({"name": line[1], "size": float(line[2]),
                               "overhead": float(line[3]), "cost": float(line[4])})
            elif key == "limit":
                limit = float(line[1])
            elif key == "expect":
                expect = ([int(v) for v in line[1:-1]], float(line[-1]))
            elif key in ("alloc", "free"):
                events.append((key, float(line[1])))
            elif key == "path":
                events.append(("path",))
            else:
                events.append((key, int(line[1])))
    return arrays, events, limit, expect
